// Schedules of many independent queues laid out back to back, and of one
// short queue, each computed inside LDS where it fits.
//
// Every queue is scheduled as the drained min-heap of Algorithm 1 (MinHeap
// Construction): ids ascending by (priority, length, id), each request's wait
// the exclusive prefix of the service times ahead of it (Eq. 1 with all
// arrivals equal), and exact per-class totals. Ids are local to the queue.
//
// Launch sequence of the batched call (the caller's stream, no host round
// trip):
//   b_plan    validates the offsets, zeroes the totals of empty queues, files
//             every queue of more than 256 requests into the work list of its
//             size class and schedules the others itself, one wave per queue
//   b_medium  queues of 257 .. 4096 requests, one 256-thread workgroup each
//   b_wide    queues of 4097 .. 16384 requests, plus every shorter queue whose
//             key does not fit a 32-bit element (the two kernels above hand
//             those on), one 1024-thread workgroup each on 64-bit elements
//   b_long    queues of more than 16384 requests: one segmented LSD radix
//             sort over all of them, in a cooperative launch
// The medium and wide work lists are split into kSubLists segments, each
// with an entry counter and a grab counter in a line of its own: the
// planner files a chunk's queues into the segment of the chunk's index
// modulo kSubLists, and a workgroup starts on the segment of its XCD
// (blockIdx % 8), takes queues from it, and moves on to the others when it
// is empty, so queues of ragged sizes spread evenly over the grid. One
// counter for a whole list would serialise the filing atomics of every
// planner workgroup and the grabs of every workgroup. The short queues of
// the planner need no such grabs: each chunk's are few and similar.
//
// Inside a workgroup a queue of m requests is loaded once (coalesced rounds
// of 64), its live key bits (priority - pmin, length - lmin) are found by a
// min/max reduction, and every request becomes one element: key above the
// local id. LSD passes over D-bit digits rank each round of 64 elements per
// wave by ballot matching of the digit bits (the width is a compile-time
// constant), turn the per-wave digit counters into positions, and permute
// the elements through an LDS stage. The exclusive length scan of the
// sorted queue gives the waits, the sorted order is class-major, so per-lane
// runs of one class give the class totals. 5 bytes are read and 12 written
// per request: the queue never leaves LDS.
#include <hip/hip_cooperative_groups.h>

#include <type_traits>

#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

namespace cg = cooperative_groups;

__device__ __forceinline__ int wave_index() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

// ---- work lists ----------------------------------------------------------------

// Request range of work item s: queue s of the batch, or the single queue.
__device__ __forceinline__ void queue_bounds(const BArgs& a, int64_t s, int64_t& base,
                                             int64_t& m) {
  if (a.offsets) {
    base = a.offsets[s];
    m = a.offsets[s + 1] - base;
  } else {
    base = 0;
    m = a.n_single;
  }
}

// First slot in a.lists of segment j of list L (medium or wide), or of the
// long list.
__device__ __forceinline__ int64_t list_base(const BArgs& a, int L, int j) {
  return L == kListLong ? 2 * kSubLists * a.seg_cap
                        : ((int64_t)(L - kListMedium) * kSubLists + j) * a.seg_cap;
}

// The segment of list L that the slot k of a.lists lies in.
__device__ __forceinline__ int segment_of(const BArgs& a, int L, int64_t k) {
  return (int)((k - list_base(a, L, 0)) / a.seg_cap);
}

// Batch i of segment j holds its entries i*B .. i*B + B - 1. Grabbers (a
// wave or a workgroup, per_wg of them per workgroup) on XCD j (blockIdx % 8)
// serve segment j first: grabber li of them takes batch li with no atomic;
// later batches come from the segment's counter, offset by the number of its
// grabbers, then from the other segments' counters (a grabber whose first
// batch is past its segment's end goes straight to those). Called by one
// lane, with the segments' entry counts n; `state` starts at -1. Returns the
// slot in a.lists of the batch's first entry (the others follow) or a
// negative value when done.
__device__ __forceinline__ uint32_t grabbers_on(int j, int per_wg) {
  const int g = (int)gridDim.x;
  return j < g ? (uint32_t)(((g - 1 - j) / kSubLists + 1) * per_wg) : 0u;
}

template <int B>
__device__ int64_t next_batch(const BArgs& a, int L, const uint32_t* n, int per_wg, uint32_t li,
                              int& state) {
  const int j0 = (int)(blockIdx.x & (kSubLists - 1));
  if (state < 0) {
    state = 0;
    const uint64_t k = (uint64_t)li * B;
    if (k < n[j0]) return list_base(a, L, j0) + (int64_t)k;
  }
  while (state < kSubLists) {
    const int j = (j0 + state) & (kSubLists - 1);
    const uint32_t free = grabbers_on(j, per_wg);  // batches taken without an atomic
    // the hint saves the atomic on a segment another grabber found empty
    if ((uint64_t)free * B < n[j] && !__hip_atomic_load(&a.ctl->empty[L][j], __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT)) {
      const uint32_t i = free + atomicAdd(&a.grab[L * kSubLists + j].next, 1u);
      const uint64_t k = (uint64_t)i * B;
      if (k < n[j]) return list_base(a, L, j) + (int64_t)k;
      __hip_atomic_store(&a.ctl->empty[L][j], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    ++state;
  }
  return -1;
}

// Appends queue s to segment j of list L (the segment of the chunk it came from).
__device__ __forceinline__ void hand_on(const BArgs& a, int L, int j, int64_t s) {
  const uint32_t pos = atomicAdd(&a.grab[L * kSubLists + j].count, 1u);
  a.lists[list_base(a, L, j) + pos] = (uint32_t)s;
}

// ---- one queue in LDS ------------------------------------------------------------

constexpr uint32_t kClsCopies = 8;  // copies of the class sums (a power of two)

// LDS of a group of NW waves that schedules one queue of at most NW*64*R
// requests with D-bit digits on elements of type ET.
template <int NW, int R, int D, typename ET>
struct GroupLds {
  static constexpr int CAP = NW * kWave * R;
  static constexpr int NB = 1 << D;
  ET stage[CAP];
  uint16_t cnt[NW][NB];  // per-wave digit counters, then per-wave digit positions
  uint64_t cls[256];     // wait sums of the queue's classes (class - pmin)
  uint32_t red[4][NW];   // range reduction
  uint64_t wtot[NW];     // per-wave sums
  uint32_t scan[NW + 1];
  int64_t next;          // next work item of the workgroup
};

template <int NW>
__device__ __forceinline__ void group_sync() {
  if constexpr (NW == 1) {
    // one wave: its LDS operations complete in order; keep the compiler from
    // moving accesses across this point and wait for the outstanding ones
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
  } else {
    block_sync();
  }
}

// Exclusive scan of one u32 per thread of the group (t = thread in group).
template <int NW>
__device__ __forceinline__ uint32_t group_excl_scan_u32(uint32_t v, uint32_t* scratch) {
  if constexpr (NW == 1) {
    return wave_incl_scan_u32(v) - v;
  } else {
    uint32_t total;
    return block_excl_scan_u32<NW * kWave>(v, scratch, total);
  }
}

// Wave reductions through DPP lane moves (no LDS traffic): row_shr steps
// within rows of 16 lanes, then row_bcast:15 and row_bcast:31 across rows;
// lanes whose source is outside the row (or masked off) take the identity.
// The result is read from lane 63.
#define SEMSCHED_DPP_REDUCE(NAME, OP, IDENT)                                                  \
  __device__ __forceinline__ uint32_t NAME(uint32_t v) {                                      \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x111, 0xf, 0xf, false)); \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x112, 0xf, 0xf, false)); \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x114, 0xf, 0xf, false)); \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x118, 0xf, 0xf, false)); \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x142, 0xa, 0xf, false)); \
    v = OP(v, (uint32_t)__builtin_amdgcn_update_dpp((int)(IDENT), (int)v, 0x143, 0xc, 0xf, false)); \
    return (uint32_t)__builtin_amdgcn_readlane((int)v, kWave - 1);                             \
  }
__device__ __forceinline__ uint32_t op_min(uint32_t a, uint32_t b) { return min(a, b); }
__device__ __forceinline__ uint32_t op_max(uint32_t a, uint32_t b) { return max(a, b); }
__device__ __forceinline__ uint32_t op_add(uint32_t a, uint32_t b) { return a + b; }
SEMSCHED_DPP_REDUCE(wave_rmin, op_min, 0xffffffffu)
SEMSCHED_DPP_REDUCE(wave_rmax, op_max, 0u)
SEMSCHED_DPP_REDUCE(wave_radd, op_add, 0u)
#undef SEMSCHED_DPP_REDUCE

// Wave sum of 64-bit values in three limbs of 22, 22 and 20 bits (each limb's
// sum over 64 lanes stays below 2^28), exact modulo 2^64.
__device__ __forceinline__ uint64_t wave_rsum_u64(uint64_t v) {
  const uint64_t a = wave_radd((uint32_t)v & 0x3fffffu);
  const uint64_t b = wave_radd((uint32_t)(v >> 22) & 0x3fffffu);
  const uint64_t c = wave_radd((uint32_t)(v >> 44));
  return a + (b << 22) + (c << 44);
}

// Wave sum of values below 2^40.
__device__ __forceinline__ uint64_t wave_sum_u40(uint64_t v) {
  return last_lane_u64(wave_incl_scan_u40(v));
}

// Wave sum of arbitrary 64-bit values (wrapping).
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  return last_lane_u64(wave_incl_scan_u64(v));
}

// Clears this wave's NB u16 counters with 64-bit stores.
template <int NB>
__device__ __forceinline__ void clear_counters(uint16_t* cnt) {
  u64_alias* c64 = reinterpret_cast<u64_alias*>(cnt);
  constexpr int WORDS = NB / 4;
  if constexpr (WORDS >= kWave) {
#pragma unroll
    for (int i = 0; i < WORDS / kWave; ++i) c64[i * kWave + lane_id()] = 0;
  } else {
    if (lane_id() < WORDS) c64[lane_id()] = 0;
  }
}

// Per-wave digit counters -> per-wave positions: on return cnt[v][b] is the
// position, in the group's digit-sorted order, of wave v's first element of
// digit b (digits ascending, waves ascending within a digit). t = thread in
// the group.
template <int NW, int NB>
__device__ __forceinline__ void digit_positions(uint16_t (*cnt)[NB], uint32_t* scratch, int t) {
  constexpr int NT = NW * kWave;
  constexpr int OWN = NB >= NT ? NB / NT : 1;
  constexpr int OWNERS = NB / OWN;
  const bool owner = OWNERS >= NT || t < OWNERS;
  uint32_t c[OWN][NW], tot[OWN];
  uint32_t local = 0;
#pragma unroll
  for (int i = 0; i < OWN; ++i) {
    tot[i] = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      c[i][v] = owner ? (uint32_t)cnt[v][t * OWN + i] : 0u;
      tot[i] += c[i][v];
    }
    local += tot[i];
  }
  uint32_t ex = group_excl_scan_u32<NW>(local, scratch);
  if (owner) {
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      uint32_t run = ex;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        cnt[v][t * OWN + i] = (uint16_t)run;
        run += c[i][v];
      }
      ex += tot[i];
    }
  }
  group_sync<NW>();
}

// Calls f(std::integral_constant<int, B>) for the B = nb in 1 .. NBITS
// (nb uniform), so that the ranking of a pass matches a compile-time number
// of digit bits.
template <int NBITS, typename F>
__device__ __forceinline__ void with_bits(uint32_t nb, F&& f) {
  if constexpr (NBITS >= 1) {
    if (nb == NBITS) {
      f(std::integral_constant<int, NBITS>{});
      return;
    }
    with_bits<NBITS - 1>(nb, f);
  }
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// A value every lane holds, stated as such to the compiler (so that it lives
// in scalar registers and branches on it are scalar).
__device__ __forceinline__ uint32_t uni(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}
__device__ __forceinline__ int64_t uni64(int64_t v) {
  const uint32_t lo = uni((uint32_t)v);
  const uint32_t hi = uni((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Buffer resource over `bytes` bytes at `base`: loads past the end return 0
// and stores past the end are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_over(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000 /* 32-bit data format, gfx9 */);
}

// Loads the requests of a queue of m requests held by a group of NW waves:
// element r of wave w's lane is request w*64*kr + r*64 + lane (rounds of 64
// consecutive requests, coalesced), kr = ceil(m / (NW*64)). Past the end the
// values read as 0.
template <int NW, int R>
__device__ __forceinline__ void load_queue(const BArgs& a, int64_t base, int m, int w,
                                           uint32_t (&pv)[R], uint32_t (&lv)[R]) {
  constexpr int NT = NW * kWave;
  base = uni64(base);
  m = (int)uni((uint32_t)m);
  const int kr = (m + NT - 1) / NT;
  const int j0 = w * kWave * kr + lane_id();
  const __amdgpu_buffer_rsrc_t rp = buffer_over(a.priority + base, (uint32_t)m);
  const __amdgpu_buffer_rsrc_t rl = buffer_over(a.length + base, 4u * (uint32_t)m);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < kr) {
      pv[r] = __builtin_amdgcn_raw_buffer_load_b8(rp, j0 + r * kWave, 0, 0);
      lv[r] = __builtin_amdgcn_raw_buffer_load_b32(rl, 4 * (j0 + r * kWave), 0, 0);
    }
  }
}

// Schedules queue s (requests base .. base+m-1, 1 <= m <= NW*64*R) from its
// loaded requests with the NW waves of a group; w = wave in the group, t =
// thread in the group. Element: key << IDB | local id, key = (priority -
// pmin) << wl | (length - lmin) over the live bits only. The passes split
// the key's bits evenly, at most D bits each. Returns false, having written
// nothing, when the key does not fit ET (the caller hands the queue on).
template <int NW, int R, int IDB, int D, typename ET>
__device__ bool schedule_loaded(const BArgs& a, int64_t s, int64_t base, int m,
                                const uint32_t (&pv)[R], const uint32_t (&lv)[R],
                                GroupLds<NW, R, D, ET>& sh, int w, int t) {
  constexpr int NT = NW * kWave;
  constexpr int NB = 1 << D;
  constexpr uint32_t EBITS = 8 * sizeof(ET);
  constexpr bool WIDE = sizeof(ET) == 8;
  const int lane = lane_id();
  s = uni64(s);
  base = uni64(base);
  m = (int)uni((uint32_t)m);
  const int kr = (m + NT - 1) / NT;  // rounds per wave (uniform)
  const int wb = w * kWave * kr;     // this wave's first position
  const int j0 = wb + lane;          // this lane's position in round 0

  // ---- ranges and validation (past the end: 0, neutral for max) --------------------
  uint32_t lmin = 0xffffffffu, lmax = 0, pmin = 0xffu, pmax = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < kr) {
      const bool valid = j0 + r * kWave < m;
      lmin = min(lmin, valid ? lv[r] : 0xffffffffu);
      lmax = max(lmax, lv[r]);
      pmin = min(pmin, valid ? pv[r] : 0xffu);
      pmax = max(pmax, pv[r]);
    }
  }
  lmin = wave_rmin(lmin);
  lmax = wave_rmax(lmax);
  pmin = wave_rmin(pmin);
  pmax = wave_rmax(pmax);
  if constexpr (NW > 1) {
    if (lane == 0) {
      sh.red[0][w] = lmin;
      sh.red[1][w] = lmax;
      sh.red[2][w] = pmin;
      sh.red[3][w] = pmax;
    }
    group_sync<NW>();
    lmin = 0xffffffffu;
    lmax = 0;
    pmin = 0xffu;
    pmax = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      lmin = min(lmin, sh.red[0][v]);
      lmax = max(lmax, sh.red[1][v]);
      pmin = min(pmin, sh.red[2][v]);
      pmax = max(pmax, sh.red[3][v]);
    }
  }
  lmin = uni(lmin);
  lmax = uni(lmax);
  pmin = uni(pmin);
  pmax = uni(pmax);
  // a negative length is above 2^31 as u32, so it shows in lmax
  if ((lmax >> 31) | (pmax >= (uint32_t)a.num_classes)) {
    if (t == 0) atomicOr(a.flags, kFlagRange);
    return true;
  }
  const uint32_t wl = bit_width32(lmax - lmin);
  const uint32_t kb = wl + bit_width32(pmax - pmin);
  if (kb + IDB > EBITS) return false;
  const uint32_t P = pmax - pmin + 1;
  // class sums in kClsCopies copies (lane % kClsCopies) when they fit, so that
  // the lanes of a round that change class together spread over that many
  // LDS addresses
  const uint32_t K = P * kClsCopies <= 256 ? kClsCopies : 1u;
  for (uint32_t c = t; c < P * K; c += NT) sh.cls[c] = 0;

  // ---- elements (past the end: all ones, the last digit of every pass; those
  // elements come last in the input, so they stay last) ---------------------------
  ET e[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < kr) {
      const int j = j0 + r * kWave;
      const ET key = ((ET)(pv[r] - pmin) << wl) | (ET)(lv[r] - lmin);
      e[r] = j < m ? ((key << IDB) | (ET)j) : ~(ET)0;
    }
  }

  // ---- LSD passes over the live key bits, in LDS ----------------------------------
  const uint32_t npass = (kb + D - 1) / D;
  const uint32_t bpp = npass ? (kb + npass - 1) / npass : 0;  // bits per pass
  uint16_t* mycnt = sh.cnt[w];
  for (uint32_t q = 0; q < npass; ++q) {
    const uint32_t shift = IDB + q * bpp;
    const uint32_t nb = min(bpp, kb - q * bpp);
    clear_counters<NB>(mycnt);
    uint32_t dg[R], rk[R];
    // A wave alone ranks with the pass's bit count compiled in (a form per
    // width); a workgroup matches its full digit width D in one form, since
    // more forms cost it registers and occupancy.
    if constexpr (NW > 1) {
      // Every lane's digit has zeros above its nb live bits, so matching all
      // D bits finds the same peers, unrolled at compile time with no loop
      // over the bits (a second, narrower form would cost registers).
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (r < kr) {
          dg[r] = (uint32_t)(e[r] >> shift) & ((1u << nb) - 1u);
          rk[r] = rank_round_c<D>(dg[r], mycnt);
        }
      }
    } else
    with_bits<D>(nb, [&](auto bits) {
      constexpr int NBITS = decltype(bits)::value;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (r < kr) {
          dg[r] = (uint32_t)(e[r] >> shift) & ((1u << NBITS) - 1u);
          rk[r] = rank_round_c<NBITS>(dg[r], mycnt);
        }
      }
    });
    group_sync<NW>();
    digit_positions<NW, NB>(sh.cnt, sh.scan, t);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r < kr) {
        sh.stage[rk[r] + mycnt[dg[r]]] = e[r];
      }
    }
    group_sync<NW>();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r < kr) {
        e[r] = sh.stage[j0 + r * kWave];
      }
    }
  }

  // ---- waits: exclusive scan of the lengths in schedule order -----------------------
  // Scanned as length - lmin (below 2^wl); the lmin part of a wait is lmin
  // times its position, whose lane part is added once and round part per round.
  const uint32_t lmask = wl ? (uint32_t)((1ull << wl) - 1) : 0u;
  uint32_t lo[R];
  uint64_t lsum = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < kr) {
      lo[r] = j0 + r * kWave < m ? (uint32_t)(e[r] >> IDB) & lmask : 0u;
      lsum += lo[r];
    }
  }
  uint64_t run = 0;  // uniform: length sum of the positions before this round
  if constexpr (NW > 1) {
    const uint64_t wsum = wave_rsum_u64(lsum);
    if (lane == 0) sh.wtot[w] = wsum;
    group_sync<NW>();
    for (int v = 0; v < w; ++v) run += sh.wtot[v];  // (w is uniform)
  }
  const uint64_t lane_part = (uint64_t)lmin * (uint32_t)j0;
  const uint64_t round_part = (uint64_t)lmin * kWave;
  const uint32_t idmask = (1u << IDB) - 1;
  const uint32_t cshift = IDB + wl;
  const __amdgpu_buffer_rsrc_t ro = buffer_over(a.order + base, 4u * (uint32_t)m);
  const __amdgpu_buffer_rsrc_t rw = buffer_over(a.wait + base, 8u * (uint32_t)m);
  int cur = -1;
  uint64_t acc = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < kr) {
      const int j = j0 + r * kWave;
      uint64_t ex, rtot;
      if constexpr (WIDE) {
        const uint64_t incl = wave_incl_scan_len(lo[r]);  // lengths up to 2^31
        ex = incl - lo[r];
        rtot = last_lane_u64(incl);
      } else {
        const uint32_t incl = wave_incl_scan_u32(lo[r]);  // 64 values below 2^24
        ex = incl - lo[r];
        rtot = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
      }
      const uint64_t wt = run + lane_part + ex;
      run += rtot + round_part;
      // past the end the buffer range check drops the stores
      __builtin_amdgcn_raw_buffer_store_b32((uint32_t)e[r] & idmask, ro, 4 * j, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{(uint32_t)wt, (uint32_t)(wt >> 32)}, rw, 8 * j,
                                            0, 0);
      if (j < m) {
        const int cls = (int)(uint32_t)(e[r] >> cshift);  // class - pmin
        if (cls != cur) {  // a lane's positions increase, so its classes do not decrease
          if (cur >= 0)
            atomicAdd(reinterpret_cast<unsigned long long*>(&sh.cls[cur * K + (lane & (K - 1))]),
                      acc);
          cur = cls;
          acc = 0;
        }
        acc += wt;  // a queue's waits add up to less than 2^59
      }
    }
  }
  if (cur >= 0)
    atomicAdd(reinterpret_cast<unsigned long long*>(&sh.cls[cur * K + (lane & (K - 1))]), acc);
  group_sync<NW>();

  // ---- totals of the queue: exact, and below 2^59, so the high words are 0 ------
  const int64_t C1 = 1 + a.num_classes;
  uint64_t* tot = a.totals + 2 * s * C1;
  for (int c = t; c < a.num_classes; c += NT) {
    uint64_t v = 0;
    if ((uint32_t)c >= pmin && (uint32_t)c <= pmax)
      for (uint32_t k = 0; k < K; ++k) v += sh.cls[(c - pmin) * K + k];
    tot[2 * (1 + c)] = v;
    tot[2 * (1 + c) + 1] = 0;
  }
  // the queue's total, the sum of its classes' sums, by the first wave alone
  if (w == 0) {
    uint64_t part = 0;
    for (uint32_t c = lane; c < P * K; c += kWave) part += sh.cls[c];
    part = wave_rsum_u64(part);
    if (lane == 0) {
      tot[0] = part;
      tot[1] = 0;
    }
  }
  return true;
}

template <int NW, int R, int IDB, int D, typename ET>
__device__ bool schedule_in_lds(const BArgs& a, int64_t s, int64_t base, int m,
                                GroupLds<NW, R, D, ET>& sh, int w, int t) {
  uint32_t pv[R], lv[R];
  load_queue<NW, R>(a, base, m, w, pv, lv);
  return schedule_loaded<NW, R, IDB, D, ET>(a, s, base, m, pv, lv, sh, w, t);
}

// ---- size-class kernels ----------------------------------------------------------

// ---- planner, and the queues of at most 256 requests ---------------------------
// Every workgroup takes chunks of `chunk` consecutive queues (the host sizes
// chunks so that every resident workgroup gets about one). Its threads read
// the queues' offsets, check them, zero the totals of empty queues and file
// every queue into a list by size: queues of at most 256 requests into a list
// in LDS that the workgroup's 4 waves then schedule themselves, one queue per
// wave at a time, round robin (no workgroup barrier, and the inputs of a
// wave's next queue load while it schedules the current one); longer queues
// into the global work lists of the other kernels (one atomic per list and
// chunk, on the chunk's segment, reserves their room).
constexpr int kPlanThreads = 256;
constexpr int kPlanWaves = kPlanThreads / kWave;
using TinyLds = GroupLds<1, 4, 8, uint32_t>;

// Eight waves per SIMD (at most 64 registers, and LDS for eight workgroups
// per CU): the planner's one-wave queues are bound by instruction issue and
// latency, and the eighth wave was worth 18 % on 65,536 queues of 256.
__global__ __launch_bounds__(kPlanThreads, 8) void b_plan(BArgs a, int chunk) {
  __shared__ uint32_t lst[kLists][kPlanChunk];
  __shared__ uint32_t lcnt[kLists], lbase[kLists];
  __shared__ unsigned long long llong;
  __shared__ TinyLds tl[kPlanWaves];
  const int t = threadIdx.x;
  const int w = wave_index();
  const int lane = lane_id();
  const int64_t S = a.num_segments;
  const int64_t C1 = 1 + a.num_classes;
  // The chunk's segment of the medium and wide lists: chunk c is planned by
  // workgroup c % gridDim.x, and the grid is a multiple of kSubLists or has
  // one chunk per workgroup, so this is c % kSubLists.
  const int seg = (int)(blockIdx.x & (kSubLists - 1));
  for (int64_t c0 = (int64_t)blockIdx.x * chunk; c0 < S; c0 += (int64_t)gridDim.x * chunk) {
    if (t < kLists) lcnt[t] = 0;
    if (t == 0) llong = 0;
    __syncthreads();
    for (int k = t; k < chunk; k += kPlanThreads) {
      const int64_t s = c0 + k;
      if (s >= S) break;
      const int64_t o0 = a.offsets[s];
      const int64_t m = a.offsets[s + 1] - o0;
      if ((s == 0 && o0 != 0) || m < 0 || m > INT32_MAX) {
        atomicOr(a.flags, kFlagInval);
        continue;
      }
      if (m == 0) {
        uint64_t* tot = a.totals + 2 * s * C1;
        for (int64_t c = 0; c < 2 * C1; ++c) tot[c] = 0;
        continue;
      }
      const int L = m <= kSegTinyCap     ? kListTiny
                    : m <= kSegMediumCap ? kListMedium
                    : m <= kSegLargeCap  ? kListWide
                                         : kListLong;
      if (L == kListLong && a.long_cap == 0) {  // no room for long queues
        atomicOr(a.flags, kFlagInval);
        continue;
      }
      const uint32_t slot = atomicAdd(&lcnt[L], 1u);
      lst[L][slot] = (uint32_t)s;
      if (L == kListLong) atomicAdd(&llong, (unsigned long long)m);
    }
    __syncthreads();
    if (t > kListTiny && t < kLists && lcnt[t])
      lbase[t] = atomicAdd(t == kListLong ? &a.ctl->count[kListLong]
                                          : &a.grab[t * kSubLists + seg].count,
                           lcnt[t]);
    if (t == 0 && llong)
      atomicAdd(reinterpret_cast<unsigned long long*>(&a.ctl->long_elems), llong);
    __syncthreads();
    for (int L = kListTiny + 1; L < kLists; ++L)
      for (uint32_t i = t; i < lcnt[L]; i += kPlanThreads)
        a.lists[list_base(a, L, seg) + lbase[L] + i] = lst[L][i];

    // the chunk's queues of at most 256 requests, wave w taking every 4th
    const uint32_t nt = lcnt[kListTiny];
    uint32_t i = (uint32_t)w;
    int64_t s = -1, base = 0, m = 0;
    uint32_t pv[4], lv[4], pn[4], ln[4];
    auto bounds = [&](uint32_t at, int64_t& qs, int64_t& qb, int64_t& qm) {
      qs = uni(lst[kListTiny][at]);
      qb = uni64(a.offsets[qs]);
      qm = uni64(a.offsets[qs + 1]) - qb;
    };
    if (i < nt) {
      bounds(i, s, base, m);
      load_queue<1, 4>(a, base, (int)m, 0, pv, lv);
    }
    while (i < nt) {
      // the inputs of this wave's next queue load while this one is scheduled
      const uint32_t i1 = i + kPlanWaves;
      int64_t s1 = -1, base1 = 0, m1 = 0;
      if (i1 < nt) {
        bounds(i1, s1, base1, m1);
        load_queue<1, 4>(a, base1, (int)m1, 0, pn, ln);
      }
      if (!schedule_loaded<1, 4, 8, 8, uint32_t>(a, s, base, (int)m, pv, lv, tl[w], 0, lane))
        if (lane == 0) hand_on(a, kListWide, seg, s);
      i = i1;
      s = s1;
      base = base1;
      m = m1;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pv[r] = pn[r];
        lv[r] = ln[r];
      }
    }
    __syncthreads();  // the chunk's lists are done with
  }
}

// Queues of 257 .. 4096 requests: one 256-thread workgroup each, digits of
// at most 7 bits. A workgroup matches all D bits of every pass, so the bits
// matched per request are D times the passes: 14 for keys of up to 14 bits
// (8 classes and lengths spanning less than 2^11), where 10-bit digits match
// 20 and 8-bit ones 16; keys of 15 .. 20 bits take three passes (21 bits, one
// more than two 10-bit passes).
using MediumLds = GroupLds<4, 16, 7, uint32_t>;

// Queues of up to 16384 requests with any key: one 1024-thread workgroup each,
// 64-bit elements. Also the single-queue call for n <= 16384.
constexpr int kWideThreads = 1024;
using WideLds = GroupLds<16, 16, 8, uint64_t>;

// Workgroup loop over one list: thread 0 grabs, the workgroup schedules.
// The grab of the next queue is issued before the current one is scheduled.
template <int NW, int R, int IDB, int D, typename ET>
__device__ void block_list_loop(const BArgs& a, int L, GroupLds<NW, R, D, ET>& sh) {
  const int t = threadIdx.x;
  const int w = wave_index();
  const uint32_t li = blockIdx.x / kSubLists;
  int state = -1;
  // the segments' entry counts (final: the kernels before this one filed
  // them), read once by the grabbing thread
  __shared__ uint32_t n[kSubLists];
  if (t == 0) {
    uint32_t c[kSubLists];
#pragma unroll
    for (int j = 0; j < kSubLists; ++j) c[j] = a.grab[L * kSubLists + j].count;
#pragma unroll
    for (int j = 0; j < kSubLists; ++j) n[j] = c[j];
    sh.next = next_batch<1>(a, L, n, 1, li, state);
  }
  block_sync();
  int64_t k = sh.next;
  while (k >= 0) {
    block_sync();  // every thread has read sh.next
    if (t == 0) sh.next = next_batch<1>(a, L, n, 1, li, state);
    const int64_t s = a.lists[k];
    int64_t base, m;
    queue_bounds(a, s, base, m);
    if (!schedule_in_lds<NW, R, IDB, D, ET>(a, s, base, (int)m, sh, w, t))
      if (t == 0) hand_on(a, kListWide, segment_of(a, L, k), s);
    block_sync();
    k = sh.next;
  }
}

// Five waves per SIMD (at most 96 registers): 6 % faster on 16,384 ragged
// queues than the four that 113 registers allowed (six spill).
__global__ __launch_bounds__(256, 5) void b_medium(BArgs a) {
  __shared__ MediumLds sh;
  block_list_loop<4, 16, 12, 7, uint32_t>(a, kListMedium, sh);
}

__global__ __launch_bounds__(kWideThreads) void b_wide(BArgs a) {
  __shared__ WideLds sh;
  if (!a.offsets) {  // the single queue
    if (blockIdx.x == 0 && a.n_single > 0) {
      if (!schedule_in_lds<16, 16, 14, 8, uint64_t>(a, 0, 0, (int)a.n_single, sh,
                                                     wave_index(), threadIdx.x))
        if (threadIdx.x == 0) atomicOr(a.flags, kFlagDevice);  // (cannot happen: 39 + 14 bits)
    }
    return;
  }
  block_list_loop<16, 16, 14, 8, uint64_t>(a, kListWide, sh);
}

// ---- segmented sort of the long queues --------------------------------------------
// All queues of more than 16384 requests at once. They are cut into tiles of
// kLongTile requests (a tile never spans two queues); the key of a request is
// (priority - pmin) << wl | (length - lmin) with the ranges of all long
// queues together, and the queue a tile belongs to is not part of the key:
// digit offsets are scanned per queue over its own tiles. The key's live
// bits are split evenly over passes of at most 10 bits; when the key and the
// request's index in its queue fit 64 bits, the index rides below the key in
// one element. Per pass: count every tile's digits, scan the counts per
// queue and digit over the queue's tiles (plus the queue's digit bases),
// scatter every tile stably. Then the waits: every tile's length sum, the exclusive scan of
// those per queue, and every tile's own scan, with exact 128-bit class
// totals. Grid-wide phases are separated by grid syncs; the launch is
// cooperative, so every workgroup is resident.
constexpr int kLT = 512;
constexpr int kLW = kLT / kWave;
constexpr int kLR = kLongTile / kLT;  // rounds per thread
constexpr int kLB = 1 << kLongDigitBits;  // digits of a pass
constexpr int kLO = kLB / kLT;            // digits per thread (consecutive)
constexpr int kCD = kLongColDigits;       // digits of a column item
constexpr int kCR = 512;                  // rows of a column item's block
constexpr int kCS = kLT / kCD;            // row segments of a block (a thread each per digit)
constexpr int kCSR = kCR / kCS;           // rows of a segment

struct LongLds {
  uint16_t cnt[kLW][kLB];
  uint32_t hrow[kLB];
  uint32_t dstart[kLB];  // start of each digit's run in the staged tile
  union {
    struct {  // the scatter's tile, staged in digit order
      uint64_t key[kLongTile];
      uint32_t id[kLongTile];
    } st;
    uint32_t acnt[kLW][kLB];  // the counting phase's per-wave counts
    struct {  // a column item's block of rows (padded rows), its segments' sums
      uint32_t v[kCR][kCD + 1];
      uint32_t seg[kCS][kCD];
    } col;
  } u;
  uint64_t clo[256], chi[256];
  uint64_t part[kLW + 1];
  uint32_t part32[kLW + 1];
  uint32_t red[4][kLW];
};

// Waits for every outstanding global load and store of the wave (s_waitcnt
// with vmcnt 0; expcnt and lgkmcnt at their maxima, so not waited for). At
// the top of a tile loop whose next tile is loaded ahead: loads and stores
// share that counter, and with the previous tile's stores still pending the
// compiler's own wait at the first use of a loaded value waits for all of
// them, the next tile's loads too; after this wait it places none.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Tile t of the long queues, found by a binary search over the first tiles
// of the K queues (in long-list order). Its chain of dependent loads is paid
// once per call: phase R stores the result in a.tdesc for the later phases.
__device__ LongTileDesc long_tile(const BArgs& a, uint32_t t, uint32_t K) {
  uint32_t k = 0, hi = K;  // tstart[k] <= t < tstart[hi]
  while (hi - k > 1) {
    const uint32_t mid = (k + hi) / 2;
    if (a.tstart[mid] <= t) k = mid;
    else hi = mid;
  }
  LongTileDesc x;
  const uint32_t r0 = a.tstart[k];
  x.s = a.lists[list_base(a, kListLong, 0) + k];
  const int64_t base = a.offsets[x.s];
  const int64_t m = a.offsets[x.s + 1] - base;
  x.lo = (t - r0) * (uint32_t)kLongTile;  // (below m < 2^31)
  x.cnt = (int32_t)min((int64_t)kLongTile, m - (int64_t)x.lo);
  x.first = base + x.lo;
  x.at = a.lbase[k] + x.lo;
  x.item0 = a.istart[k];
  x.rows = a.tstart[k + 1] - r0;
  return x;
}

// Tile tt's descriptor, or an empty tile past the last one.
__device__ __forceinline__ LongTileDesc tile_or_empty(const BArgs& a, uint32_t tt,
                                                      uint32_t ntiles) {
  LongTileDesc x = {};
  if (tt < ntiles) x = a.tdesc[tt];
  return x;
}

__global__ __launch_bounds__(kLT) void b_long(BArgs a) {
  __shared__ LongLds sh;
  cg::grid_group grid = cg::this_grid();
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = wave_index();
  const uint32_t K = a.ctl->count[kListLong];
  if (K == 0) return;  // (uniform: written by earlier kernels)
  if (a.ctl->long_elems > a.long_cap) {
    if (blockIdx.x == 0 && t == 0) atomicOr(a.flags, kFlagInval);  // workspace too small
    return;
  }
  const int64_t C1 = 1 + a.num_classes;

  // ---- phase 0: queue starts and first tiles (workgroup 0); zero the totals --------
  if (blockIdx.x == 0) {
    uint64_t carry_e = 0;
    uint32_t carry_t = 0, carry_i = 0;
    for (uint32_t k0 = 0; k0 < K; k0 += kLT) {
      const uint32_t k = k0 + t;
      uint64_t m = 0;
      if (k < K) {
        const int64_t s = a.lists[list_base(a, kListLong, 0) + k];
        m = (uint64_t)(a.offsets[s + 1] - a.offsets[s]);
      }
      const uint32_t tiles = (uint32_t)((m + kLongTile - 1) / kLongTile);
      const uint32_t items = k < K ? (tiles <= kLongRowsFew ? 1u : (uint32_t)(kLB / kCD)) : 0u;
      uint64_t tot_e;
      uint32_t tot_t, tot_i;
      const uint64_t ex_e = block_excl_scan_u64<kLT>(m, sh.part, tot_e);
      const uint32_t ex_t = block_excl_scan_u32<kLT>(tiles, sh.part32, tot_t);
      const uint32_t ex_i = block_excl_scan_u32<kLT>(items, sh.part32, tot_i);
      if (k < K) {
        a.lbase[k] = carry_e + ex_e;
        a.tstart[k] = carry_t + ex_t;
        a.istart[k] = carry_i + ex_i;
      }
      carry_e += tot_e;
      carry_t += tot_t;
      carry_i += tot_i;
    }
    if (t == 0) {
      a.lbase[K] = carry_e;
      a.tstart[K] = carry_t;
      a.istart[K] = carry_i;
      if (carry_t > a.max_tiles) atomicOr(a.flags, kFlagInval);  // (cannot happen)
      a.ctl->ranges[0] = 0xffu;
      a.ctl->ranges[1] = 0;
      a.ctl->ranges[2] = 0xffffffffu;
      a.ctl->ranges[3] = 0;
      a.ctl->ranges[4] = 0;
    }
  }
  for (int64_t i = (int64_t)blockIdx.x * kLT + t; i < (int64_t)K * 2 * C1;
       i += (int64_t)gridDim.x * kLT) {
    const int64_t s = a.lists[list_base(a, kListLong, 0) + i / (2 * C1)];
    a.totals[2 * s * C1 + i % (2 * C1)] = 0;
  }
  grid.sync();
  const uint32_t ntiles = a.tstart[K];
  const uint32_t nitems = a.istart[K];

  // ---- phase R: ranges and validation of all long queues --------------------------
  // Reduced over the workgroup's tiles first, then one atomic per range word
  // and workgroup, skipped when it would not change the word: atomics on one
  // line serialise, and one per wave and tile queued thousands on it.
  {
    uint32_t lmin = 0xffffffffu, lmax = 0, pmin = 0xffu, pmax = 0, bad = 0, mmax = 0;
    for (uint32_t tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
      const LongTileDesc x = long_tile(a, tt, K);
      if (t == 0) a.tdesc[tt] = x;
      mmax = max(mmax, x.lo + (uint32_t)x.cnt);  // (uniform) the queue's size at its last tile
      if (x.lo == 0) {  // (uniform) the queue's first tile: map its digit-offset items
        const uint32_t nit = x.rows <= kLongRowsFew ? 1u : (uint32_t)(kLB / kCD);
        for (uint32_t j = t; j < nit; j += kLT) a.imap[x.item0 + j] = tt;
      }
      uint32_t p[kLR];
      int32_t l[kLR];
#pragma unroll
      for (int r = 0; r < kLR; ++r) {  // (every load issued before the first use)
        const int i = r * kLT + t;
        p[r] = 0;
        l[r] = 0;
        if (i < x.cnt) {
          p[r] = a.priority[x.first + i];
          l[r] = a.length[x.first + i];
        }
      }
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        if (r * kLT + t < x.cnt) {
          bad |= (l[r] < 0) | ((int)p[r] >= a.num_classes);
          lmin = min(lmin, (uint32_t)l[r]);
          lmax = max(lmax, (uint32_t)l[r]);
          pmin = min(pmin, p[r]);
          pmax = max(pmax, p[r]);
        }
      }
    }
    lmin = wave_min_u32(lmin);
    lmax = wave_max_u32(lmax);
    pmin = wave_min_u32(pmin);
    pmax = wave_max_u32(pmax);
    bad = wave_or_u32(bad);
    if (lane == 0) {
      if (bad) atomicOr(a.flags, kFlagRange);
      sh.red[0][w] = pmin;
      sh.red[1][w] = pmax;
      sh.red[2][w] = lmin;
      sh.red[3][w] = lmax;
    }
    block_sync();
    if (t == 0) {
      for (int v = 1; v < kLW; ++v) {
        pmin = min(pmin, sh.red[0][v]);
        pmax = max(pmax, sh.red[1][v]);
        lmin = min(lmin, sh.red[2][v]);
        lmax = max(lmax, sh.red[3][v]);
      }
      uint32_t* rg = a.ctl->ranges;
      if (pmin < load_agent(rg + 0)) atomicMin(rg + 0, pmin);
      if (pmax > load_agent(rg + 1)) atomicMax(rg + 1, pmax);
      if (lmin < load_agent(rg + 2)) atomicMin(rg + 2, lmin);
      if (lmax > load_agent(rg + 3)) atomicMax(rg + 3, lmax);
      if (mmax > load_agent(rg + 4)) atomicMax(rg + 4, mmax);  // (mmax: the same in every thread)
    }
  }
  grid.sync();
  // Every workgroup decides the same: nothing writes the flags from here on
  // (the earlier kernels and phases R and 0 are done), so no workgroup can
  // leave while others wait at a later grid sync.
  if (__hip_atomic_load(a.flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
  auto range = [&](int i) {
    return __hip_atomic_load(&a.ctl->ranges[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  const uint32_t pmin = range(0), pmax = range(1);
  const uint32_t lmin = range(2), lmax = range(3);
  const uint32_t wl = bit_width32(lmax - lmin);
  const uint32_t kb = wl + bit_width32(pmax - pmin);
  const int npass = kb ? (int)((kb + kLongDigitBits - 1) / kLongDigitBits) : 1;
  // the key's bits split evenly over the passes: longer runs per digit in
  // the scatter than a full first digit and a short last one
  const uint32_t dbits = (kb + npass - 1) / npass;
  const uint32_t dmask = (1u << dbits) - 1;
  const uint64_t lmask = wl ? ((1ull << wl) - 1) : 0;
  // When the key and the request's index in its queue fit 64 bits together,
  // the index rides in the element's low ib bits (8 bytes per element
  // between the passes instead of a key and a separate id); else ib = 0.
  const uint32_t idb = bit_width32(range(4) - 1);
  const bool packed = kb + idb <= 64;
  const uint32_t ib = packed ? idb : 0u;
  const uint64_t idmask = (1ull << ib) - 1;

  // element r of this thread in tile x: request x.lo + w*64*kLR + r*64 + lane
  // (with_ids false: the ids are not read, for the counting phase)
  auto load_elems = [&](const LongTileDesc& x, int q, uint64_t (&key)[kLR],
                        uint32_t (&id)[kLR], bool with_ids) {
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = w * kWave * kLR + r * kWave + lane;
      key[r] = ~0ull;
      id[r] = 0;
      if (i < x.cnt) {
        if (q == 0) {
          const uint32_t p = a.priority[x.first + i];
          const uint32_t l = (uint32_t)a.length[x.first + i];
          id[r] = x.lo + (uint32_t)i;
          key[r] = ((((uint64_t)(p - pmin) << wl) | (uint64_t)(l - lmin)) << ib) |
                   (packed ? id[r] : 0u);
        } else {
          key[r] = a.keys[(q - 1) & 1][x.at + i];
          if (with_ids && !packed) id[r] = a.ids[(q - 1) & 1][x.at + i];
        }
      }
    }
  };

  for (int q = 0; q < npass; ++q) {
    const uint32_t shift = ib + dbits * q;
    // ---- phase A: digit counts of every tile ----------------------------------------
    // (the workgroup's next tile is loaded while this one is counted)
    {
    LongTileDesc x = tile_or_empty(a, blockIdx.x, ntiles);
    uint64_t key[kLR];
    uint32_t id[kLR];
    load_elems(x, q, key, id, false);
    for (uint32_t tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
      wait_vmem();
      const LongTileDesc xn = tile_or_empty(a, tt + gridDim.x, ntiles);
      uint64_t nkey[kLR];
      uint32_t nid[kLR];
      load_elems(xn, q, nkey, nid, false);
      // (counts only: one LDS add per request into the wave's own table)
      uint32_t* mine = sh.u.acnt[w];
      for (int b = lane; b < kLB; b += kWave) mine[b] = 0;
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        const int i = w * kWave * kLR + r * kWave + lane;
        if (i < x.cnt) atomicAdd(&mine[(uint32_t)(key[r] >> shift) & dmask], 1u);
      }
      block_sync();
#pragma unroll
      for (int o = 0; o < kLO; ++o) {
        const int d = kLO * t + o;
        uint32_t c = 0;
#pragma unroll
        for (int v = 0; v < kLW; ++v) c += sh.u.acnt[v][d];
        a.hist[(size_t)tt * kLB + d] = c;
      }
      block_sync();
      x = xn;
#pragma unroll
      for (int r = 0; r < kLR; ++r) key[r] = nkey[r];
    }
    }
    grid.sync();
    // ---- phase B: per queue and digit, offsets over the queue's tiles ----------------
    // A queue of few tiles is one work item: each thread runs down the
    // columns of its kLO digits and the digit bases are added at once. A
    // queue of many tiles is kLB / kCD items of kCD digits each, whose
    // columns are scanned together down the queue's tiles; its digit totals
    // go to qtot and the digit bases are added by the scatter (phase C).
    for (uint32_t it = blockIdx.x; it < nitems; it += gridDim.x) {
      const uint32_t r0 = a.imap[it];  // the queue's first tile
      const LongTileDesc y = a.tdesc[r0];
      const uint32_t r1 = r0 + y.rows;
      if (y.rows <= kLongRowsFew) {
        uint32_t tot[kLO], sum = 0;
#pragma unroll
        for (int o = 0; o < kLO; ++o) {
          tot[o] = 0;
          for (uint32_t row = r0; row < r1; ++row)
            tot[o] += a.hist[(size_t)row * kLB + kLO * t + o];
          sum += tot[o];
        }
        uint32_t total;
        uint32_t run = block_excl_scan_u32<kLT>(sum, sh.part32, total);
#pragma unroll
        for (int o = 0; o < kLO; ++o) {
          uint32_t r = run;
          for (uint32_t row = r0; row < r1; ++row) {
            uint32_t* h = a.hist + (size_t)row * kLB + kLO * t + o;
            const uint32_t c = *h;
            *h = r;
            r += c;
          }
          run += tot[o];
        }
      } else {
        // kCD digits from d0: blocks of kCR rows are loaded coalesced into
        // LDS, each thread scans kCSR rows of one digit, a thread per digit
        // scans the segments' sums (carrying the earlier blocks' totals), and
        // the offsets go back coalesced
        const uint32_t d0 = (it - y.item0) * kCD;
        uint32_t carry = 0;  // (threads t < kCD: digit d0 + t)
        for (uint32_t row0 = r0; row0 < r1; row0 += kCR) {
          uint32_t* hb = a.hist + (size_t)row0 * kLB + d0;  // (uniform)
          const uint32_t nr = min(r1 - row0, (uint32_t)kCR);
          // the thread index through an empty asm: the offsets below are
          // formed here, not hoisted out of every loop around this one (they
          // would hold registers through the other phases)
          int tv = t;
          asm volatile("" : "+v"(tv));
#pragma unroll
          for (int j = 0; j < kCR * kCD / kLT; ++j) {
            const int v = j * kLT + tv;
            sh.u.col.v[v / kCD][v % kCD] =
                (uint32_t)(v / kCD) < nr ? hb[(v / kCD) * kLB + v % kCD] : 0u;
          }
          block_sync();
          {
            const int dd = tv % kCD, sg = tv / kCD;
            uint32_t run = 0;
#pragma unroll
            for (int k = 0; k < kCSR; ++k) {
              const uint32_t c = sh.u.col.v[sg * kCSR + k][dd];
              sh.u.col.v[sg * kCSR + k][dd] = run;
              run += c;
            }
            sh.u.col.seg[sg][dd] = run;
          }
          block_sync();
          if (t < kCD) {
#pragma unroll 8
            for (int g = 0; g < kCS; ++g) {
              const uint32_t c = sh.u.col.seg[g][t];
              sh.u.col.seg[g][t] = carry;
              carry += c;
            }
          }
          block_sync();
#pragma unroll
          for (int j = 0; j < kCR * kCD / kLT; ++j) {
            const int v = j * kLT + tv;
            if ((uint32_t)(v / kCD) < nr)
              hb[(v / kCD) * kLB + v % kCD] =
                  sh.u.col.v[v / kCD][v % kCD] + sh.u.col.seg[(v / kCD) / kCSR][v % kCD];
          }
          block_sync();
        }
        if (t < kCD) a.qtot[(size_t)it * kCD + t] = carry;
      }
    }
    grid.sync();
    // ---- phase C: stable scatter of every tile ----------------------------------------
    // (the workgroup's next tile, its digit offsets and its queue's digit
    // totals are loaded while this one is placed and written)
    {
    LongTileDesc x = tile_or_empty(a, blockIdx.x, ntiles);
    uint64_t key[kLR];
    uint32_t id[kLR], hv[kLO], qv[kLO];
    auto load_offsets = [&](const LongTileDesc& y, uint32_t ty, uint32_t (&h)[kLO],
                            uint32_t (&c)[kLO]) {
#pragma unroll
      for (int o = 0; o < kLO; ++o) {
        h[o] = y.cnt > 0 ? a.hist[(size_t)ty * kLB + kLO * t + o] : 0u;
        c[o] = y.rows > kLongRowsFew ? a.qtot[(size_t)y.item0 * kCD + kLO * t + o] : 0u;
      }
    };
    load_elems(x, q, key, id, true);
    load_offsets(x, blockIdx.x, hv, qv);
    for (uint32_t tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
      wait_vmem();
      uint32_t dg[kLR], rk[kLR];
      uint32_t dbase[kLO] = {};  // queues of many tiles: the digits' bases in the queue
      if (x.rows > kLongRowsFew) {  // (uniform)
        uint32_t sum = 0;
#pragma unroll
        for (int o = 0; o < kLO; ++o) sum += qv[o];
        uint32_t total;
        uint32_t run = block_excl_scan_u32<kLT>(sum, sh.part32, total);
#pragma unroll
        for (int o = 0; o < kLO; ++o) {
          dbase[o] = run;
          run += qv[o];
        }
      }
#pragma unroll
      for (int o = 0; o < kLO; ++o) sh.hrow[kLO * t + o] = hv[o] + dbase[o];
      clear_counters<kLB>(sh.cnt[w]);
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        dg[r] = (uint32_t)(key[r] >> shift) & dmask;
        rk[r] = rank_round_c<kLongDigitBits>(dg[r], sh.cnt[w]);
      }
      const uint32_t tn = tt + gridDim.x;
      const LongTileDesc xn = tile_or_empty(a, tn, ntiles);
      uint64_t nkey[kLR];
      uint32_t nid[kLR];
      load_elems(xn, q, nkey, nid, true);
      load_offsets(xn, tn, hv, qv);
      block_sync();
      // owners: the waves' offsets within each digit, then the digits'
      // starts in the tile (elements past the end count in the last digit
      // and rank after its real ones, so they shift no real position)
      uint32_t tot[kLO], sum = 0;
#pragma unroll
      for (int o = 0; o < kLO; ++o) {
        const int d = kLO * t + o;
        uint32_t run = 0;
#pragma unroll
        for (int v = 0; v < kLW; ++v) {
          const uint32_t c = sh.cnt[v][d];
          sh.cnt[v][d] = (uint16_t)run;
          run += c;
        }
        tot[o] = run;
        sum += run;
      }
      {
        uint32_t total;
        uint32_t st = block_excl_scan_u32<kLT>(sum, sh.part32, total);  // (barriers)
#pragma unroll
        for (int o = 0; o < kLO; ++o) {
          sh.dstart[kLO * t + o] = st;
          st += tot[o];
        }
      }
      block_sync();
      // stage the tile in digit order, then write it out in runs per digit
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        const int i = w * kWave * kLR + r * kWave + lane;
        if (i < x.cnt) {
          const uint32_t j = sh.dstart[dg[r]] + sh.cnt[w][dg[r]] + rk[r];
          sh.u.st.key[j] = key[r];
          if (!packed) sh.u.st.id[j] = id[r];
        }
      }
      block_sync();
      uint64_t* kout = a.keys[q & 1] + (x.at - x.lo);  // the queue's first element
      uint32_t* iout = a.ids[q & 1] + (x.at - x.lo);
      for (int j = t; j < x.cnt; j += kLT) {
        const uint64_t k = sh.u.st.key[j];
        const uint32_t d = (uint32_t)(k >> shift) & dmask;
        const uint32_t at = sh.hrow[d] + (uint32_t)(j - (int)sh.dstart[d]);
        kout[at] = k;
        if (!packed) iout[at] = sh.u.st.id[j];
      }
      block_sync();
      x = xn;
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        key[r] = nkey[r];
        id[r] = nid[r];
      }
    }
    }
    grid.sync();
  }

  // ---- waits and totals of the sorted queues ----------------------------------------
  const uint64_t* skey = a.keys[(npass - 1) & 1];
  const uint32_t* sid = a.ids[(npass - 1) & 1];
  // phase D1: length sum of every tile
  // (the workgroup's next tile is loaded while this one is summed)
  {
  auto load_keys = [&](const LongTileDesc& y, uint64_t (&v)[kLR]) {
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = r * kLT + t;
      v[r] = i < y.cnt ? skey[y.at + i] : 0;
    }
  };
  LongTileDesc x = tile_or_empty(a, blockIdx.x, ntiles);
  uint64_t v[kLR];
  load_keys(x, v);
  for (uint32_t tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
    wait_vmem();
    const LongTileDesc xn = tile_or_empty(a, tt + gridDim.x, ntiles);
    uint64_t nv[kLR];
    load_keys(xn, nv);
    uint64_t s = 0;
#pragma unroll
    for (int r = 0; r < kLR; ++r) s += r * kLT + t < x.cnt ? ((v[r] >> ib) & lmask) + lmin : 0;
    s = wave_sum_u64(s);
    if (lane == 0) sh.part[w] = s;
    block_sync();
    if (t == 0) {
      uint64_t sum = 0;
      for (int u = 0; u < kLW; ++u) sum += sh.part[u];
      a.tsum[tt] = sum;
    }
    block_sync();
    x = xn;
#pragma unroll
    for (int r = 0; r < kLR; ++r) v[r] = nv[r];
  }
  }
  grid.sync();
  // phase D2: per queue, exclusive scan of its tiles' sums
  for (uint32_t k = blockIdx.x; k < K; k += gridDim.x) {
    const uint32_t r0 = a.tstart[k], r1 = a.tstart[k + 1];
    uint64_t carry = 0;
    for (uint32_t row0 = r0; row0 < r1; row0 += kLT) {
      const uint32_t row = row0 + t;
      const uint64_t v = row < r1 ? a.tsum[row] : 0ull;
      uint64_t total;
      const uint64_t ex = block_excl_scan_u64<kLT>(v, sh.part, total);
      if (row < r1) a.tsum[row] = carry + ex;
      carry += total;
    }
  }
  grid.sync();
  // phase D3: order, waits and class totals of every tile. The class sums
  // of the workgroup's consecutive tiles of one queue add up in LDS and go
  // to the queue's totals when the queue changes and at the end (one atomic
  // per class and one for the total at each such flush).
  const uint32_t P = pmax - pmin + 1;
  int64_t cur_s = -1;  // (uniform) the queue whose sums the LDS totals hold
  auto flush = [&]() {
    block_sync();  // every lane's sums are in
    uint64_t* tot = a.totals + 2 * cur_s * C1;
    for (uint32_t c = t; c < P; c += kLT) {
      const U128 v = {sh.clo[c], sh.chi[c]};
      if (v.lo | v.hi) atomic_add128(tot + 2 * (1 + pmin + c), tot + 2 * (1 + pmin + c) + 1, v);
    }
    if (t == 0) {
      U128 g = {0, 0};
      for (uint32_t c = 0; c < P; ++c) add128(g, U128{sh.clo[c], sh.chi[c]});
      if (g.lo | g.hi) atomic_add128(tot, tot + 1, g);
    }
    block_sync();  // the sums are read
    for (uint32_t c = t; c < P; c += kLT) sh.clo[c] = sh.chi[c] = 0;
  };
  for (uint32_t c = t; c < P; c += kLT) sh.clo[c] = sh.chi[c] = 0;
  // (the workgroup's next tile and its wait base are loaded while this one
  // is written)
  auto load_sorted = [&](const LongTileDesc& y, uint32_t ty, uint64_t (&key)[kLR],
                         uint32_t (&id)[kLR], uint64_t& wbase) {
    // (packed: the ids are taken from the keys where they are stored, so
    // that no load waits for the one before it)
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = w * kWave * kLR + r * kWave + lane;
      key[r] = i < y.cnt ? skey[y.at + i] : 0ull;
    }
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = w * kWave * kLR + r * kWave + lane;
      id[r] = !packed && i < y.cnt ? sid[y.at + i] : 0u;
    }
    wbase = y.cnt > 0 ? a.tsum[ty] : 0;
  };
  LongTileDesc x = tile_or_empty(a, blockIdx.x, ntiles);
  uint64_t key[kLR], wbase;
  uint32_t id[kLR];
  load_sorted(x, blockIdx.x, key, id, wbase);
  for (uint32_t tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
    wait_vmem();
    if (x.s != cur_s) {  // (uniform)
      if (cur_s >= 0) flush();
      cur_s = x.s;
    }
    block_sync();  // the totals are cleared
    uint32_t len[kLR];
    uint64_t mine = 0;
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = w * kWave * kLR + r * kWave + lane;
      len[r] = i < x.cnt ? (uint32_t)(((key[r] >> ib) & lmask) + lmin) : 0u;
      mine += len[r];
    }
    const uint32_t tn = tt + gridDim.x;
    const LongTileDesc xn = tile_or_empty(a, tn, ntiles);
    uint64_t nkey[kLR], nwbase;
    uint32_t nid[kLR];
    load_sorted(xn, tn, nkey, nid, nwbase);
    const uint64_t wsum = wave_sum_u64(mine);
    if (lane == 0) sh.part[w] = wsum;
    block_sync();
    uint64_t run = wbase;
    for (int v = 0; v < w; ++v) run += sh.part[v];  // (w is uniform)
    int cur = -1;
    U128 acc = {0, 0};
    const int64_t out0 = x.first;
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      const int i = w * kWave * kLR + r * kWave + lane;
      const uint64_t incl = wave_incl_scan_len(len[r]);
      const uint64_t wt = run + incl - len[r];
      run += last_lane_u64(incl);
      if (i < x.cnt) {
        a.order[out0 + i] = (int32_t)(packed ? (uint32_t)(key[r] & idmask) : id[r]);
        a.wait[out0 + i] = (int64_t)wt;
        const int cls = (int)(key[r] >> (ib + wl));
        if (cls != cur) {
          if (cur >= 0) atomic_add128(&sh.clo[cur], &sh.chi[cur], acc);
          cur = cls;
          acc = U128{0, 0};
        }
        add128(acc, wt);
      }
    }
    if (cur >= 0) atomic_add128(&sh.clo[cur], &sh.chi[cur], acc);
    block_sync();  // (sh.part is read; the next tile writes it)
    x = xn;
    wbase = nwbase;
#pragma unroll
    for (int r = 0; r < kLR; ++r) {
      key[r] = nkey[r];
      id[r] = nid[r];
    }
  }
  if (cur_s >= 0) flush();  // (uniform)
}

// ---- host side -------------------------------------------------------------------

template <typename K>
int resident(K kernel, int threads) {
  int dev = 0, cus = 256, occ = 1;
  if (hipGetDevice(&dev) == hipSuccess) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) cus = prop.multiProcessorCount;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, reinterpret_cast<const void*>(kernel),
                                                   threads, 0) != hipSuccess ||
      occ < 1)
    occ = 1;
  return cus * occ;
}

int grid_for(int resident_blocks, int64_t want) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(resident_blocks, want));
}

}  // namespace

uint32_t long_max_tiles(uint64_t long_cap, int64_t num_segments) {
  // every long queue has more than kSegLargeCap requests
  const uint64_t queues = std::min<uint64_t>((uint64_t)std::max<int64_t>(num_segments, 0),
                                             long_cap / (kSegLargeCap + 1));
  return (uint32_t)((long_cap + kLongTile - 1) / kLongTile + queues + 1);
}

hipError_t launch_single_lds(const BArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(b_wide, dim3(1), dim3(kWideThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_batched(const BArgs& a, hipStream_t st) {
  static const int r_plan = resident(b_plan, kPlanThreads);
  static const int r_medium = resident(b_medium, 256);
  static const int r_wide = resident(b_wide, kWideThreads);
  static const int r_long = resident(b_long, kLT);
  const int64_t S = a.num_segments;
  // chunks of about S / (resident planner workgroups) queues, at most
  // kPlanChunk; a grid of one workgroup per chunk, or else a multiple of
  // kSubLists (the planner files chunk c into list segment c % kSubLists)
  const int r8 = std::max(kSubLists, r_plan / kSubLists * kSubLists);
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(kPlanChunk, (S + r8 - 1) / r8));
  hipLaunchKernelGGL(b_plan, dim3(grid_for(r8, (S + chunk - 1) / chunk)), dim3(kPlanThreads), 0,
                     st, a, (int)chunk);
  hipLaunchKernelGGL(b_medium, dim3(grid_for(r_medium, S)), dim3(256), 0, st, a);
  hipLaunchKernelGGL(b_wide, dim3(grid_for(r_wide, S)), dim3(kWideThreads), 0, st, a);
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  if (a.long_cap > 0) {
    const int g = grid_for(r_long, (int64_t)long_max_tiles(a.long_cap, S));
    BArgs copy = a;
    void* args[] = {&copy};
    const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(b_long),
                                                    dim3(g), dim3(kLT), args, 0, st);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

}  // namespace semsched
