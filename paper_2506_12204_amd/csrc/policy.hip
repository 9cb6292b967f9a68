// Comparison policies of the request-spike experiments (Section 4): first
// come first served (arrival order), shortest job first (predicted length,
// then id) and highest-priority job first (urgency rank, then id). Waits are
// the exclusive prefix of the lengths in the policy's order and the totals
// are split by each request's own rank, as for the semantic order.
//
// Every kernel gives each wave one range of kPolRange consecutive positions
// (64 rounds of 64 lanes); a block's four waves are independent. With at most
// kRegClasses ranks every lane keeps its own per-class sums in registers
// (one compare and two selects per class and element) and the wave reduces
// them once per range. With more ranks the sums are formed once per round
// for each rank present among the round's lanes (a uniform loop: pick a
// lane's rank, ballot its peers, reduce them) and kept in lanes: class c in
// lane c % 64 of register set c / 64. The two forms are separate kernels
// (registers are allocated per kernel); both are launched and the one that
// does not fit the class count returns at once.
//
//   p_range    largest rank (the class count P = largest + 1)
//   FCFS       f_sums: length sum of every range, length check, largest rank;
//              f_scan: exclusive scan of the range sums;
//              f_write: order[k] = k, wait = range offset + in-range prefix
//   HPJF       h_count: per range and class, count and length sum;
//              h_scan: per class, exclusive scans of both over the ranges;
//              h_scatter: a stable counting sort by rank, each element at
//              (class start + range offset + rank among its class in the
//              range) with wait = the same prefix of lengths
//   SJF        the semantic kernels with every rank read as 0 (the order by
//              (length, id)); where their compact layout has room, the
//              elements carry the caller's ranks and the final pass splits
//              the totals by them (s_classes and p_total then return at
//              once); else s_classes: per-class sums of the waits with each
//              position's rank gathered through its id
//   p_total    adds the per-block class sums of the last pass: totals
#include <algorithm>

#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int PT = 256;                // threads of the range kernels (4 waves)
constexpr int kWaves = PT / kWave;
constexpr int kRounds = kPolRange / kWave;  // 64 rounds per range
constexpr int kBatch = 8;              // rounds loaded together
constexpr int kBatches = kRounds / kBatch;
constexpr int ST = 1024;               // threads of the scan kernels
static_assert(kRounds % kBatch == 0, "whole batches per range");

typedef const __attribute__((address_space(4))) uint64_t ConstU64;
typedef const __attribute__((address_space(4))) uint32_t ConstU32;

__device__ __forceinline__ int64_t wave_index() {
  return (int64_t)blockIdx.x * kWaves + __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

__device__ __forceinline__ uint32_t class_count(const PolArgs& a) {
  return *((ConstU32*)a.pmax) + 1u;  // (written by p_range, a kernel before)
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return (uint64_t)hi << 32 | lo;
}

// Uniform 64 x 32 -> 128-bit product plus a 64-bit addend.
__device__ __forceinline__ U128 mul_add(uint64_t x, uint32_t k, uint64_t add) {
  U128 r = {x * k, __umul64hi(x, (uint64_t)k)};
  add128(r, add);
  return r;
}

// 256 per-class values held in lanes: class c in lane c % 64 of set c / 64.
// SETS = 1 when every rank is below 64. The class index and the value added
// are uniform across the wave.
template <int SETS, typename T>
struct LaneTab {
  T v[SETS];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < SETS; ++i) v[i] = 0;
  }
  __device__ __forceinline__ T pick(int s) const {
    T x = v[0];
#pragma unroll
    for (int i = 1; i < SETS; ++i) x = s == i ? v[i] : x;
    return x;
  }
  __device__ __forceinline__ T get(uint32_t c) const {
    const T x = pick((int)(c >> 6));
    if constexpr (sizeof(T) == 8) return readlane_u64(x, (int)(c & 63));
    else return (T)__builtin_amdgcn_readlane((int)x, (int)(c & 63));
  }
  __device__ __forceinline__ void add(uint32_t c, T d) {
    const bool me = lane_id() == (int)(c & 63);
#pragma unroll
    for (int i = 0; i < SETS; ++i) v[i] += (me && (int)(c >> 6) == i) ? d : (T)0;
  }
};

// Exact 128-bit per-class sums in lanes.
template <int SETS>
struct LaneAcc {
  LaneTab<SETS, uint64_t> lo, hi;
  __device__ __forceinline__ void zero() {
    lo.zero();
    hi.zero();
  }
  __device__ __forceinline__ void add(uint32_t c, const U128& d) {
    const bool me = lane_id() == (int)(c & 63);
#pragma unroll
    for (int i = 0; i < SETS; ++i) {
      const bool on = me && (int)(c >> 6) == i;
      const uint64_t dl = on ? d.lo : 0, dh = on ? d.hi : 0;
      lo.v[i] += dl;
      hi.v[i] += dh + (lo.v[i] < dl ? 1u : 0u);
    }
  }
};

constexpr int kRegClasses = 8;  // up to this many ranks, per-lane class sums in registers

// Per-lane sums of 64-bit values (below 2^62) for classes c < PB, kept as the
// sums of their low and high 32-bit halves: a lane adds at most kRounds
// values per range, so each half-sum stays below 2^38.
template <int PB>
struct RegSums {
  uint64_t lo[PB], hi[PB];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int c = 0; c < PB; ++c) lo[c] = hi[c] = 0;
  }
  __device__ __forceinline__ void add(uint32_t cls, uint64_t v, uint32_t P) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      if (c < (int)P) {
        const bool on = cls == (uint32_t)c;
        lo[c] += on ? (uint32_t)v : 0u;
        hi[c] += on ? (uint32_t)(v >> 32) : 0u;
      }
    }
  }
};

// Per-lane element counts and length sums for classes c < PB.
template <int PB>
struct RegCounts {
  uint32_t cnt[PB];
  uint64_t len[PB];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      cnt[c] = 0;
      len[c] = 0;
    }
  }
  __device__ __forceinline__ void add(uint32_t cls, uint32_t l, bool live, uint32_t P) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      if (c < (int)P) {
        const bool on = live && cls == (uint32_t)c;
        cnt[c] += on ? 1u : 0u;
        len[c] += on ? l : 0u;
      }
    }
  }
};

// Calls f(c, peers) once for every distinct rank c among the lanes of `live`
// (`peers` = the live lanes holding c). All 64 lanes must be active.
template <typename F>
__device__ __forceinline__ void for_each_class(uint32_t cls, uint64_t live, F&& f) {
  uint64_t rem = live;
  while (rem) {
    const int l0 = __builtin_ctzll(rem);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)cls, l0);
    const uint64_t peers = __ballot(cls == c) & live;
    f(c, peers);
    rem &= ~peers;
  }
}

__device__ __forceinline__ bool in_mask(uint64_t m) { return (m >> lane_id()) & 1ull; }

// Sum over the wave of values below 2^40 (per-lane prefixes of a round).
__device__ __forceinline__ uint64_t wave_sum_u40(uint64_t v) {
  return readlane_u64(wave_incl_scan_u40(v), 63);
}

// The block's class sums: every wave adds its lanes into LDS, then the first
// P threads store them as the block's row of the partial table.
struct PartShared {
  uint64_t lo[256], hi[256];
};

template <int SETS>
__device__ __forceinline__ void store_lane_acc(const LaneAcc<SETS>& acc, PartShared& sh) {
#pragma unroll
  for (int s = 0; s < SETS; ++s) {
    const U128 v = {acc.lo.v[s], acc.hi.v[s]};
    const int c = s * kWave + lane_id();
    if (v.lo | v.hi) atomic_add128(sh.lo + c, sh.hi + c, v);
  }
}

// Lane 0 adds a wave-uniform class sum into the block's LDS table.
__device__ __forceinline__ void add_partial(PartShared& sh, uint32_t c, const U128& v) {
  if (lane_id() == 0 && (v.lo | v.hi)) atomic_add128(sh.lo + c, sh.hi + c, v);
}

// The block's row of the partial table (after every wave has added its sums).
__device__ __forceinline__ void write_partials(const PolArgs& a, PartShared& sh, uint32_t P) {
  block_sync();
  const int t = threadIdx.x;
  if (t < (int)P) {
    uint64_t* row = a.part + 2 * ((uint64_t)blockIdx.x * P + t);
    row[0] = sh.lo[t];
    row[1] = sh.hi[t];
  }
}

template <int PB>
__device__ __forceinline__ void flush_sums(PartShared& sh, const RegSums<PB>& s, uint32_t P) {
#pragma unroll
  for (int c = 0; c < PB; ++c) {
    if (c < (int)P) {
      const uint64_t l = wave_sum_u40(s.lo[c]), h = wave_sum_u40(s.hi[c]);
      U128 v = {l, 0};
      add128(v, U128{h << 32, h >> 32});
      add_partial(sh, (uint32_t)c, v);
    }
  }
}

__device__ __forceinline__ void zero_partials(PartShared& sh) {
  sh.lo[threadIdx.x] = sh.hi[threadIdx.x] = 0;
  block_sync();
}

// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t max_byte(uint32_t m, uint32_t x) {
  m = max(m, x & 0xffu);
  m = max(m, (x >> 8) & 0xffu);
  m = max(m, (x >> 16) & 0xffu);
  return max(m, x >> 24);
}

// Largest rank over all requests: 16-byte loads over the aligned body,
// single bytes before and after it.
// Adds this workgroup's largest value to *dst: a wave maximum, the workgroup
// maximum in LDS, then one global atomic, skipped when *dst already holds at
// least as much (one device-scope atomic on a single word serialises at
// about 11 ns; one per wave over a 2^26-request queue took longer than the
// loads themselves). Every thread of the workgroup must call it.
__device__ __forceinline__ void group_max_to(uint32_t* dst, uint32_t m) {
  __shared__ uint32_t gmax;
  if (threadIdx.x == 0) gmax = 0;
  __syncthreads();
  m = wave_max_u32(m);
  if (lane_id() == 0 && m) atomicMax(&gmax, m);
  __syncthreads();
  if (threadIdx.x == 0 && gmax && gmax > load_agent(dst)) atomicMax(dst, gmax);
}

__global__ __launch_bounds__(PT) void p_range(PolArgs a) {
  const uintptr_t addr = reinterpret_cast<uintptr_t>(a.priority);
  const int64_t head = std::min<int64_t>(a.n, (int64_t)((16 - (addr & 15)) & 15));
  const int64_t body = (a.n - head) / 16;
  const uint4* v = reinterpret_cast<const uint4*>(a.priority + head);
  const int64_t stride = (int64_t)gridDim.x * PT;
  const int64_t t = (int64_t)blockIdx.x * PT + threadIdx.x;
  uint32_t m = 0;
  for (int64_t i = t; i < body; i += stride) {
    const uint4 x = v[i];
    m = max_byte(max_byte(max_byte(max_byte(m, x.x), x.y), x.z), x.w);
  }
  if (t < head) m = max(m, (uint32_t)a.priority[t]);
  const int64_t tail = head + body * 16;
  if (tail + t < a.n) m = max(m, (uint32_t)a.priority[tail + t]);  // (fewer than 16 left)
  group_max_to(a.pmax, m);
}

// Calls f(length, rank, live) for every element of the range starting at k0
// (kPolRange elements, in no particular order). With vec (lengths 16-byte
// and ranks 4-byte aligned) every lane loads four consecutive elements at a
// time; elements past n come with live = false. All lanes call f together.
template <typename F>
__device__ __forceinline__ void range_elements(const PolArgs& a, int64_t k0, bool vec, F&& f) {
  if (vec) {
#pragma unroll 4
    for (int r = 0; r < kRounds / 4; ++r) {
      const int64_t k = k0 + 4 * ((int64_t)r * kWave + lane_id());
      int32_t l[4];
      uint32_t p[4];
      if (k + 3 < a.n) {
        const int4 lv = *reinterpret_cast<const int4*>(a.length + k);
        const uint32_t pv = *reinterpret_cast<const uint32_t*>(a.priority + k);
        l[0] = lv.x, l[1] = lv.y, l[2] = lv.z, l[3] = lv.w;
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = (pv >> (8 * i)) & 0xffu;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t ki = min(k + i, a.n - 1);
          l[i] = a.length[ki];
          p[i] = a.priority[ki];
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) f(l[i], p[i], k + i < a.n);
    }
  } else {
#pragma unroll 16
    for (int r = 0; r < kRounds; ++r) {
      const int64_t k = k0 + r * kWave + lane_id();
      const int64_t kc = min(k, a.n - 1);
      f(a.length[kc], (uint32_t)a.priority[kc], k < a.n);
    }
  }
}

__device__ __forceinline__ bool vec_ok(const PolArgs& a) {
  return ((reinterpret_cast<uintptr_t>(a.length) & 15) | (reinterpret_cast<uintptr_t>(a.priority) & 3)) == 0;
}

// FCFS: length sum of every range and the largest rank; negative lengths
// are flagged.
__global__ __launch_bounds__(PT) void f_sums(PolArgs a, int64_t ranges) {
  const int64_t w = min(wave_index(), ranges - 1);  // (waves past the end repeat the last range)
  const bool live = wave_index() < ranges;
  const int64_t k0 = w * kPolRange;
  uint64_t s = 0;
  uint32_t m = 0;
  bool bad = false;
  // (one element per lane: this first kernel of a schedule runs while the
  // caches write back the previous schedule's output, and loading four per
  // lane did not help it)
#pragma unroll 16
  for (int r = 0; r < kRounds; ++r) {
    const int64_t k = k0 + r * kWave + lane_id();
    const int64_t kc = min(k, a.n - 1);
    const int32_t l = k < a.n ? a.length[kc] : 0;
    m = max(m, (uint32_t)a.priority[kc]);
    bad |= l < 0;
    s += (uint32_t)l;
  }
  if (__ballot(bad)) {
    if (lane_id() == 0) atomicOr(a.flags, kFlagRange);
  }
  group_max_to(a.pmax, m);
  s = readlane_u64(wave_incl_scan_u64(s), 63);
  if (lane_id() == 0 && live) a.rsum[w] = s;
}

// Exclusive scan in place of `count` contiguous values (one block; thread t
// scans the t-th chunk of ceil(count / ST) values). Chunks of up to kChunk
// values are loaded in one unrolled batch. Returns the total to every thread.
constexpr int kChunk = 16;

template <typename T>
__device__ __forceinline__ T chunk_scan(T* v, int64_t count, T* scratch) {
  const int t = threadIdx.x;
  const int64_t per = (count + ST - 1) / ST;
  const int64_t lo = min(count, t * per), hi = min(count, lo + per);
  T x[kChunk];
  T s = 0;
  if (per <= kChunk) {
#pragma unroll
    for (int i = 0; i < kChunk; ++i) x[i] = lo + i < hi ? v[lo + i] : (T)0;
#pragma unroll
    for (int i = 0; i < kChunk; ++i) s += x[i];
  } else {
    for (int64_t i = lo; i < hi; ++i) s += v[i];
  }
  T tot;
  T run;
  if constexpr (sizeof(T) == 8) run = block_excl_scan_u64<ST>(s, scratch, tot);
  else run = block_excl_scan_u32<ST>(s, scratch, tot);
  if (per <= kChunk) {
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
      if (lo + i < hi) v[lo + i] = run;
      run += x[i];
    }
  } else {
    for (int64_t i = lo; i < hi; ++i) {
      const T y = v[i];
      v[i] = run;
      run += y;
    }
  }
  return tot;
}

__global__ __launch_bounds__(ST) void f_scan(PolArgs a, int64_t ranges) {
  __shared__ uint64_t scratch[ST / kWave + 1];
  chunk_scan<uint64_t>(a.rsum, ranges, scratch);
}

// FCFS: order[k] = k, wait[k] = offset of the range + prefix inside it.
// PB > 0: per-class sums in registers (P <= PB); PB = 0: the class loop with
// lane tables of SETS sets.
template <int PB, int SETS>
__device__ __forceinline__ void fcfs_range(const PolArgs& a, int64_t w, uint32_t P,
                                           PartShared& sh) {
  RegSums<PB == 0 ? 1 : PB> rs;
  LaneAcc<SETS> acc;
  rs.zero();
  acc.zero();
  const int64_t k0 = w * kPolRange;
  uint64_t base = *((ConstU64*)(a.rsum + w));
  int32_t len[kBatch], nlen[kBatch];  // this batch, the next one
  uint8_t pri[kBatch], npri[kBatch];
  auto load = [&](int b, int32_t* l, uint8_t* p) {
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t k = min(k0 + (b * kBatch + r) * kWave + lane_id(), a.n - 1);
      l[r] = a.length[k];
      p[r] = a.priority[k];
    }
  };
  load(0, len, pri);
#pragma unroll 1
  for (int b = 0; b < kBatches; ++b) {
    load(min(b + 1, kBatches - 1), nlen, npri);  // (the last batch reloads itself)
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t kr = k0 + (b * kBatch + r) * kWave;
      const int64_t k = kr + lane_id();
      const bool live = k < a.n;
      const uint32_t lv = live ? (uint32_t)len[r] : 0u;
      const uint64_t incl = wave_incl_scan_len(lv);
      const uint64_t excl = incl - lv;
      const uint64_t wt = base + excl;
      int32_t* po = live ? a.order + k : reinterpret_cast<int32_t*>(a.sink);
      int64_t* pw = live ? a.wait + k : reinterpret_cast<int64_t*>(a.sink + 1);
      *po = (int32_t)k;
      *pw = (int64_t)wt;
      if constexpr (PB > 0) {
        rs.add((uint32_t)pri[r], live ? wt : 0, P);
      } else {
        for_each_class((uint32_t)pri[r], __ballot(live), [&](uint32_t c, uint64_t peers) {
          const uint64_t s2 = wave_sum_u40(in_mask(peers) ? excl : 0);
          acc.add(c, mul_add(base, (uint32_t)__popcll(peers), s2));
        });
      }
      base += readlane_u64(incl, 63);
    }
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      len[r] = nlen[r];
      pri[r] = npri[r];
    }
  }
  if constexpr (PB > 0) flush_sums<PB>(sh, rs, P);
  else store_lane_acc<SETS>(acc, sh);
}

template <int PB, int SETS>
__device__ __forceinline__ void fcfs_write(const PolArgs& a, int64_t ranges, PartShared& sh,
                                           uint32_t P) {
  const int64_t w = wave_index();
  if (w < ranges) fcfs_range<PB, SETS>(a, w, P, sh);
  write_partials(a, sh, P);
}

template <bool REG>
__global__ __launch_bounds__(PT) void f_write(PolArgs a, int64_t ranges) {
  __shared__ PartShared sh;
  const uint32_t P = class_count(a);
  if (REG != (P <= kRegClasses)) return;
  zero_partials(sh);
  if constexpr (REG) fcfs_write<kRegClasses, 1>(a, ranges, sh, P);
  else fcfs_write<0, 4>(a, ranges, sh, P);
}

// ---------------------------------------------------------------------------
// HPJF

// Per-class counts and length sums of one range: in registers (PB > 0) or by
// the class loop into lane tables of SETS sets.
template <int PB, int SETS>
__device__ __forceinline__ void hpjf_count(const PolArgs& a, int64_t w, int64_t ranges,
                                           uint32_t P) {
  RegCounts<PB == 0 ? 1 : PB> rc;
  LaneTab<SETS, uint32_t> cnt;
  LaneTab<SETS, uint64_t> lsum;
  rc.zero();
  cnt.zero();
  lsum.zero();
  const int64_t k0 = w * kPolRange;
  bool bad = false;
  range_elements(a, k0, vec_ok(a), [&](int32_t l, uint32_t p, bool live) {
    bad |= live && l < 0;
    const uint32_t lv = live ? (uint32_t)l : 0u;
    if constexpr (PB > 0) {
      rc.add(p, lv, live, P);
    } else {
      for_each_class(p, __ballot(live), [&](uint32_t c, uint64_t peers) {
        cnt.add(c, (uint32_t)__popcll(peers));
        lsum.add(c, readlane_u64(wave_incl_scan_len(in_mask(peers) ? lv : 0u), 63));
      });
    }
  });
  if (__ballot(bad)) {
    if (lane_id() == 0) atomicOr(a.flags, kFlagRange);
  }
  if constexpr (PB > 0) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      if (c < (int)P) {
        const uint32_t tc = (uint32_t)__builtin_amdgcn_readlane(
            (int)wave_incl_scan_u32(rc.cnt[c]), 63);
        const uint64_t tl = wave_sum_u40(rc.len[c]);  // (a lane's sum is below 2^37)
        if (lane_id() == 0) {
          a.tab_cnt[c * ranges + w] = tc;
          a.tab_len[c * ranges + w] = tl;
        }
      }
    }
  } else {
#pragma unroll
    for (int s = 0; s < SETS; ++s) {
      const uint32_t c = s * kWave + lane_id();
      if (c < P) {
        a.tab_cnt[c * ranges + w] = cnt.v[s];
        a.tab_len[c * ranges + w] = lsum.v[s];
      }
    }
  }
}

template <bool REG>
__global__ __launch_bounds__(PT) void h_count(PolArgs a, int64_t ranges) {
  const int64_t w = wave_index();
  const uint32_t P = class_count(a);
  if (w >= ranges || REG != (P <= kRegClasses)) return;
  if constexpr (REG) hpjf_count<kRegClasses, 1>(a, w, ranges, P);
  else hpjf_count<0, 4>(a, w, ranges, P);
}

// Block c: exclusive scans over the ranges of class c's counts and length
// sums (in place; the tables are class-major); the class's size and length
// total.
__global__ __launch_bounds__(ST) void h_scan(PolArgs a, int64_t ranges) {
  __shared__ uint32_t s32[ST / kWave + 1];
  __shared__ uint64_t s64[ST / kWave + 1];
  const uint32_t P = class_count(a);
  const uint32_t c = blockIdx.x;
  if (c >= P) return;
  const uint32_t tc = chunk_scan<uint32_t>(a.tab_cnt + (int64_t)c * ranges, ranges, s32);
  const uint64_t tl = chunk_scan<uint64_t>(a.tab_len + (int64_t)c * ranges, ranges, s64);
  if (threadIdx.x == 0) {
    a.ctot_cnt[c] = tc;
    a.ctot_len[c] = tl;
  }
}

// One range of the stable scatter by rank. Every lane's element goes to
// (running position of its class) + (rank among the round's lanes of that
// class) with wait = (running wait of its class) + (lengths of those lanes
// before it). PB > 0: at most PB classes with their running position and
// wait in scalar registers; a round's lanes are permuted into (class, lane)
// order, one wave scan of the permuted lengths gives every lane its prefix,
// and the prefix at the start of its class is subtracted; class sums of the
// waits in lane registers. PB = 0: the class loop over the ranks present,
// one masked scan per rank, running values and sums in lane tables.
template <int PB, int SETS>
__device__ __forceinline__ void hpjf_range(const PolArgs& a, int64_t w, int64_t ranges,
                                           uint32_t P, PartShared& sh) {
  // start of every class in this range: class start (exclusive scan of the
  // class sizes / length totals) + the range's offset inside the class
  LaneTab<SETS, uint32_t> pos;
  LaneTab<SETS, uint64_t> wb;
  uint32_t carry_c = 0;
  uint64_t carry_l = 0;
#pragma unroll
  for (int s = 0; s < SETS; ++s) {
    const uint32_t c = s * kWave + lane_id();
    const uint32_t cc = c < P ? a.ctot_cnt[c] : 0u;
    const uint64_t cl = c < P ? a.ctot_len[c] : 0u;
    const uint32_t ic = wave_incl_scan_u32(cc);
    const uint64_t il = wave_incl_scan_u64(cl);
    pos.v[s] = carry_c + ic - cc + (c < P ? a.tab_cnt[c * ranges + w] : 0u);
    wb.v[s] = carry_l + il - cl + (c < P ? a.tab_len[c * ranges + w] : 0u);
    carry_c += (uint32_t)__builtin_amdgcn_readlane((int)ic, 63);
    carry_l += readlane_u64(il, 63);
  }
  constexpr int NB = PB == 0 ? 1 : PB;
  uint32_t spos[NB];
  uint64_t swb[NB];
  if constexpr (PB > 0) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      spos[c] = (uint32_t)__builtin_amdgcn_readlane((int)pos.v[0], c);
      swb[c] = readlane_u64(wb.v[0], c);
    }
  }
  RegSums<NB> rs;
  LaneAcc<SETS> acc;
  rs.zero();
  acc.zero();
  const int64_t k0 = w * kPolRange;
  int32_t len[kBatch], nlen[kBatch];  // this batch, the next one
  uint8_t pri[kBatch], npri[kBatch];
  auto load = [&](int b, int32_t* l, uint8_t* p) {
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t k = min(k0 + (b * kBatch + r) * kWave + lane_id(), a.n - 1);
      l[r] = a.length[k];
      p[r] = a.priority[k];
    }
  };
  load(0, len, pri);
#pragma unroll 1
  for (int b = 0; b < kBatches; ++b) {
    load(min(b + 1, kBatches - 1), nlen, npri);  // (the last batch reloads itself)
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t k = k0 + (b * kBatch + r) * kWave + lane_id();
      const bool live = k < a.n;
      const uint32_t lv = live ? (uint32_t)len[r] : 0u;
      const uint32_t cls = pri[r];
      uint32_t q = 0;
      uint64_t wt = 0;
      auto place = [&](uint64_t peers, uint32_t pc, uint64_t wc, uint32_t& pnext,
                       uint64_t& wnext) {
        const bool mine = in_mask(peers);
        const uint32_t mv = mine ? lv : 0u;
        const uint64_t incl = wave_incl_scan_len(mv);
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(peers >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u));
        q = mine ? pc + rank : q;
        wt = mine ? wc + (incl - mv) : wt;
        pnext = pc + (uint32_t)__popcll(peers);
        wnext = wc + readlane_u64(incl, 63);
        return incl - mv;
      };
      const uint64_t lmask = __ballot(live);
      if constexpr (PB > 0) {
        // this lane's class: its live lanes, the live lanes of lower
        // classes, its running position and wait (lanes without an element
        // rank after every live lane, among themselves)
        uint64_t mine = ~lmask;
        uint32_t below = (uint32_t)__popcll(lmask);
        uint32_t pbase = 0;
        uint64_t wbase = 0;
        uint32_t first[PB + 1];  // (uniform) slot of each class's first lane
        uint32_t seen = 0;
#pragma unroll
        for (int c = 0; c < PB; ++c) {
          first[c] = seen;
          if (c < (int)P) {
            const bool on = live && cls == (uint32_t)c;
            const uint64_t peers = __ballot(on);
            mine = on ? peers : mine;
            below = on ? seen : below;
            pbase = on ? spos[c] : pbase;
            wbase = on ? swb[c] : wbase;
            seen += (uint32_t)__popcll(peers);
          }
        }
        first[PB] = seen;
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(mine >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mine, 0u));
        const uint32_t slot = below + rank;  // a permutation of the 64 lanes
        // lengths in (class, lane) order, their inclusive scan, read back at
        // this lane's slot and at the slot before its class
        const uint32_t sl = (uint32_t)__builtin_amdgcn_ds_permute((int)(slot * 4), (int)lv);
        const uint64_t incl = wave_incl_scan_len(sl);
        auto pull = [&](uint32_t from) {
          const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(from * 4),
                                                                     (int)(uint32_t)incl);
          const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(
              (int)(from * 4), (int)(uint32_t)(incl >> 32));
          return (uint64_t)hi << 32 | lo;
        };
        const uint64_t at = pull(slot);
        const uint64_t before = pull(below > 0 ? below - 1 : 0);
        const uint64_t ahead = below > 0 ? before : 0;  // lengths of the lower classes
        q = pbase + rank;
        wt = wbase + (at - lv - ahead);
        // running positions and waits: each class's count and length sum
        uint64_t lp = 0;  // (uniform) scan value before class c's first slot
#pragma unroll
        for (int c = 0; c < PB; ++c) {
          if (c < (int)P) {
            const uint32_t e = first[c + 1];
            const uint64_t le = e > 0 ? readlane_u64(incl, (int)e - 1) : 0;
            spos[c] += e - first[c];
            swb[c] += le - lp;
            lp = le;
          }
        }
        rs.add(cls, live ? wt : 0, P);
      } else {
        for_each_class(cls, lmask, [&](uint32_t c, uint64_t peers) {
          const uint32_t pc = pos.get(c);
          const uint64_t wc = wb.get(c);
          uint32_t pn;
          uint64_t wn;
          const uint64_t excl = place(peers, pc, wc, pn, wn);
          const uint32_t cnt = pn - pc;
          acc.add(c, mul_add(wc, cnt, wave_sum_u40(in_mask(peers) ? excl : 0)));
          pos.add(c, cnt);
          wb.add(c, wn - wc);
        });
      }
      const bool ok = live && (int64_t)q < a.n;  // (always, for consistent counts)
      int32_t* po = ok ? a.order + q : reinterpret_cast<int32_t*>(a.sink);
      int64_t* pw = ok ? a.wait + q : reinterpret_cast<int64_t*>(a.sink + 1);
      *po = (int32_t)k;
      *pw = (int64_t)wt;
    }
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      len[r] = nlen[r];
      pri[r] = npri[r];
    }
  }
  if constexpr (PB > 0) flush_sums<PB>(sh, rs, P);
  else store_lane_acc<SETS>(acc, sh);
}

template <int PB, int SETS>
__device__ __forceinline__ void hpjf_scatter(const PolArgs& a, int64_t ranges, PartShared& sh,
                                             uint32_t P) {
  const int64_t w = wave_index();
  if (w < ranges) hpjf_range<PB, SETS>(a, w, ranges, P, sh);
  write_partials(a, sh, P);
}

template <bool REG>
__global__ __launch_bounds__(PT) void h_scatter(PolArgs a, int64_t ranges) {
  __shared__ PartShared sh;
  const uint32_t P = class_count(a);
  if (REG != (P <= kRegClasses)) return;
  zero_partials(sh);
  if constexpr (REG) hpjf_scatter<kRegClasses, 1>(a, ranges, sh, P);
  else hpjf_scatter<0, 4>(a, ranges, sh, P);
}

// ---------------------------------------------------------------------------
// SJF: per-class sums of an existing schedule's waits, the rank of each
// position gathered through its id. Waits grow along the schedule, so each
// round's waits are lane 0's plus a difference below 2^37.

template <int PB, int SETS>
__device__ __forceinline__ void class_range(const PolArgs& a, int64_t w, uint32_t P,
                                            PartShared& sh) {
  RegSums<PB == 0 ? 1 : PB> rs;
  LaneAcc<SETS> acc;
  rs.zero();
  acc.zero();
  const int64_t k0 = w * kPolRange;
#pragma unroll 1
  for (int b = 0; b < kBatches; ++b) {
    int32_t id[kBatch];
    uint64_t wt[kBatch];
    uint32_t p[kBatch];
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t k = min(k0 + (b * kBatch + r) * kWave + lane_id(), a.n - 1);
      id[r] = a.order[k];
      wt[r] = (uint64_t)a.wait[k];
    }
#pragma unroll
    for (int r = 0; r < kBatch; ++r)
      p[r] = a.priority[min(max((int64_t)id[r], (int64_t)0), a.n - 1)];
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
      const int64_t k = k0 + (b * kBatch + r) * kWave + lane_id();
      const bool live = k < a.n;
      if constexpr (PB > 0) {
        rs.add(p[r], live ? wt[r] : 0, P);
      } else {
        const uint64_t w0 = readlane_u64(wt[r], 0);
        const uint64_t d = wt[r] - w0;
        for_each_class(p[r], __ballot(live), [&](uint32_t c, uint64_t peers) {
          acc.add(c, mul_add(w0, (uint32_t)__popcll(peers),
                             wave_sum_u40(in_mask(peers) ? d : 0)));
        });
      }
    }
  }
  if constexpr (PB > 0) flush_sums<PB>(sh, rs, P);
  else store_lane_acc<SETS>(acc, sh);
}

template <int PB, int SETS>
__device__ __forceinline__ void class_sums(const PolArgs& a, int64_t ranges, PartShared& sh,
                                           uint32_t P) {
  const int64_t w = wave_index();
  if (w < ranges) class_range<PB, SETS>(a, w, P, sh);
  write_partials(a, sh, P);
}

template <bool REG>
__global__ __launch_bounds__(PT) void s_classes(PolArgs a, int64_t ranges) {
  __shared__ PartShared sh;
  if (a.pay && *a.pay) return;  // the sort split the totals already
  // The sort left its own grand total; p_total adds the class sums to a
  // zero one (no other kernel touches it until p_total).
  if (REG && blockIdx.x == 0 && threadIdx.x < 2) a.totals[threadIdx.x] = 0;
  const uint32_t P = class_count(a);
  if (REG != (P <= kRegClasses)) return;
  zero_partials(sh);
  if constexpr (REG) class_sums<kRegClasses, 1>(a, ranges, sh, P);
  else class_sums<0, 4>(a, ranges, sh, P);
}

// Block c: class c's total from the blocks' partial sums (written over the
// entry); added to the grand total as well, which was zeroed before.
__global__ __launch_bounds__(PT) void p_total(PolArgs a, int64_t blocks) {
  __shared__ U128 ws[kWaves];
  if (a.pay && *a.pay) return;
  const uint32_t P = class_count(a);
  const uint32_t c = blockIdx.x;
  if (c >= P) return;
  U128 s = {0, 0};
  for (int64_t b = threadIdx.x; b < blocks; b += PT) {
    const uint64_t* row = a.part + 2 * ((uint64_t)b * P + c);
    add128(s, U128{row[0], row[1]});
  }
  s = wave_sum128(s);
  if (lane_id() == 0) ws[threadIdx.x / kWave] = s;
  block_sync();
  if (threadIdx.x == 0) {
    U128 g = {0, 0};
    for (int i = 0; i < kWaves; ++i) add128(g, ws[i]);
    a.totals[2 * (1 + c)] = g.lo;
    a.totals[2 * (1 + c) + 1] = g.hi;
    if (g.lo | g.hi) atomic_add128(a.totals, a.totals + 1, g);
  }
}

int64_t ranges_of(int64_t n) { return (n + kPolRange - 1) / kPolRange; }
int64_t blocks_of(int64_t n) { return (ranges_of(n) + kWaves - 1) / kWaves; }

hipError_t launch_p_range(const PolArgs& a, hipStream_t st) {
  const int64_t g = std::min<int64_t>((a.n + PT * 64 - 1) / (PT * 64), 1024);
  hipLaunchKernelGGL(p_range, dim3((unsigned)std::max<int64_t>(g, 1)), dim3(PT), 0, st, a);
  return hipGetLastError();
}

void mark(hipEvent_t e, hipStream_t st) {
  if (e) (void)hipEventRecord(e, st);
}

}  // namespace

int64_t policy_ranges(int64_t n) { return ranges_of(n); }
int64_t policy_blocks(int64_t n) { return blocks_of(n); }

hipError_t launch_fcfs(const PolArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after) {
  const int64_t ranges = ranges_of(a.n), blocks = blocks_of(a.n);
  hipLaunchKernelGGL(f_sums, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(f_scan, dim3(1), dim3(ST), 0, st, a, ranges);
  mark(before, st);
  hipLaunchKernelGGL(f_write<true>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(f_write<false>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  mark(after, st);
  hipLaunchKernelGGL(p_total, dim3(256), dim3(PT), 0, st, a, blocks);
  return hipGetLastError();
}

hipError_t launch_hpjf(const PolArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after) {
  const int64_t ranges = ranges_of(a.n), blocks = blocks_of(a.n);
  if (launch_p_range(a, st) != hipSuccess) return hipGetLastError();
  hipLaunchKernelGGL(h_count<true>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(h_count<false>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(h_scan, dim3(256), dim3(ST), 0, st, a, ranges);
  mark(before, st);
  hipLaunchKernelGGL(h_scatter<true>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(h_scatter<false>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  mark(after, st);
  hipLaunchKernelGGL(p_total, dim3(256), dim3(PT), 0, st, a, blocks);
  return hipGetLastError();
}

hipError_t launch_policy_range(const PolArgs& a, hipStream_t st) { return launch_p_range(a, st); }

hipError_t launch_class_totals(const PolArgs& a, hipStream_t st, hipEvent_t before,
                               hipEvent_t after) {
  const int64_t ranges = ranges_of(a.n), blocks = blocks_of(a.n);
  mark(before, st);
  hipLaunchKernelGGL(s_classes<true>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  hipLaunchKernelGGL(s_classes<false>, dim3((unsigned)blocks), dim3(PT), 0, st, a, ranges);
  mark(after, st);
  hipLaunchKernelGGL(p_total, dim3(256), dim3(PT), 0, st, a, blocks);
  return hipGetLastError();
}

}  // namespace semsched
