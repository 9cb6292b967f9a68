// Insertion of newly arrived requests into an existing schedule: the
// data-parallel form of Algorithm 1's HeapInsert under the asynchronous
// queue management of Section 3.3 (arrivals join the heap that already
// holds the earlier requests; draining it gives the schedule of all).
//
// The earlier requests 0 .. n_old-1 come as their schedule (order_old,
// wait_old); the m arrivals n_old .. n-1 are first scheduled on their own
// (the queue kernels), giving their sorted order and the prefix sums of
// their lengths. Then:
//
//   i_search  for every arrival j (in its sorted order) the number ins[j] of
//             earlier requests whose key (priority, length) is not above
//             its key (ties go to the earlier request, whose id is smaller),
//             by binary search over order_old; for every unit of kInsUnit
//             earlier entries the number of arrivals placed before its first
//             entry (the arrivals whose key is below that entry's) and the
//             classes of its first and last entries; the class starts of the
//             earlier sequence; the total length of each sequence.
//   i_merge   earlier entry k moves to k + c(k), c(k) = the number of
//             arrivals with ins[j] <= k, and its wait grows by the lengths of
//             those c(k) arrivals (their prefix sum); arrival j lands at
//             ins[j] + j with wait = (earlier wait at ins[j]) + (its wait
//             among the arrivals). Class totals are summed on the way (the
//             merged schedule is class-major, as both inputs are).
//
// Only the arrivals are sorted; every earlier entry is read and written
// once (4 + 8 bytes each way).
#include <algorithm>

#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int IT = 256;          // threads of the search kernel
constexpr int MT = 256;          // threads of the merge kernel (4 waves)
constexpr int MR = kInsUnit / kWave;  // rounds of 64 entries in a unit
constexpr int kClassSlots = 257;  // class starts (classes 0..255 and the end)
constexpr int kMaxMergeBlocks = 4096;
static_assert(MT == 256, "the merge kernel's final reduction keeps one class per thread");

// Global memory that no kernel writes while the merge kernel runs, read
// through the constant address space so that uniform loads become scalar
// loads (their completion is counted apart from the vector stores).
typedef const __attribute__((address_space(4))) uint64_t ConstU64;

// key of an earlier entry / of an arrival, both as (priority, length)
struct KeyPL {
  uint32_t p, l;
};

__device__ __forceinline__ bool key_le(KeyPL a, KeyPL b) {
  return a.p < b.p || (a.p == b.p && a.l <= b.l);
}

__device__ __forceinline__ bool key_lt(KeyPL a, KeyPL b) {
  return a.p < b.p || (a.p == b.p && a.l < b.l);
}

__device__ __forceinline__ int32_t clamp_id(int32_t id, int64_t n) {
  return (int32_t)min(max((int64_t)id, (int64_t)0), n - 1);
}

__device__ __forceinline__ KeyPL old_key(const InsArgs& a, int64_t k) {
  const int32_t id = clamp_id(a.order_old[k], a.n_old);
  return {a.priority[id], (uint32_t)a.length[id]};
}

__device__ __forceinline__ KeyPL new_key(const InsArgs& a, int64_t j) {
  const int64_t id = a.n_old + clamp_id(a.order_m[j], a.m);
  return {a.priority[id], (uint32_t)a.length[id]};
}

// Threads 0 .. m-1: ins[j]. The next units + 1: desc[u]. The next 257: class
// start c of the earlier sequence (the number of its entries with priority
// < c). One more: the two length totals.
__global__ __launch_bounds__(IT) void i_search(InsArgs a, int64_t units) {
  const int64_t i = (int64_t)blockIdx.x * IT + threadIdx.x;
  if (i < a.m) {
    const KeyPL kj = new_key(a, i);
    int64_t lo = 0, hi = a.n_old;  // upper bound: first earlier entry above kj
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (key_le(old_key(a, mid), kj)) lo = mid + 1; else hi = mid;
    }
    a.ins[i] = (uint32_t)lo;
    return;
  }
  int64_t r = i - a.m;
  if (r <= units) {
    // ins[j] <= k0 exactly when earlier entry k0 is above arrival j (the
    // earlier sequence is sorted), so c(k0) counts the arrivals below it
    const int64_t k0 = r * kInsUnit;
    uint64_t d = (uint64_t)a.m;
    if (k0 < a.n_old) {
      const KeyPL e = old_key(a, k0);
      int64_t lo = 0, hi = a.m;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (key_lt(new_key(a, mid), e)) lo = mid + 1; else hi = mid;
      }
      const uint32_t last = old_key(a, min(k0 + kInsUnit, a.n_old) - 1).p;
      d = (uint64_t)lo | (uint64_t)e.p << 32 | (uint64_t)last << 40;
    }
    a.desc[r] = d;
    return;
  }
  r -= units + 1;
  if (r < kClassSlots) {
    const uint32_t c = (uint32_t)r;
    int64_t lo = 0, hi = a.n_old;  // first entry with priority >= c
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (old_key(a, mid).p < c) lo = mid + 1; else hi = mid;
    }
    a.cs[r] = (uint32_t)lo;
    return;
  }
  if (r == kClassSlots) {
    // total lengths: last wait + last length of each sequence
    a.lsum[0] = a.n_old > 0 ? (uint64_t)a.wait_old[a.n_old - 1] + old_key(a, a.n_old - 1).l : 0;
    a.lsum[1] = a.m > 0 ? (uint64_t)a.wait_m[a.m - 1] + new_key(a, a.m - 1).l : 0;
  }
}

struct MergeShared {
  uint32_t cs[kClassSlots];   // class starts of the earlier sequence
  uint64_t clo[256], chi[256];
  U128 wsum[MT / kWave];
};

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return (uint64_t)hi << 32 | lo;
}

__device__ __forceinline__ uint64_t bpermute64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(lane << 2, (int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(lane << 2, (int)(uint32_t)(v >> 32));
  return (uint64_t)hi << 32 | lo;
}

__device__ __forceinline__ void flush(MergeShared& sh, int cur, U128& acc) {
  if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
  acc = {0, 0};
}

// One unit's inputs, loaded a unit ahead of their use.
struct UnitIn {
  int32_t id[MR];   // order_old of entries k0 + r * 64 + lane
  uint64_t w0[MR];  // their waits in the earlier schedule
  uint32_t sins;    // lane i: ins of arrival c0 + i (the unit's i-th arrival)
  uint64_t spn;     // lane i: lengths of the arrivals before c0 + i
};

// Every load is in bounds and unconditional (a fixed count per unit):
// positions past the end read the last entry instead.
__device__ __forceinline__ void load_unit(const InsArgs& a, int64_t u, uint64_t d, int lane,
                                          uint64_t lnew, UnitIn& in) {
  const int64_t k0 = u * kInsUnit;
#pragma unroll
  for (int r = 0; r < MR; ++r) {
    const int64_t k = min(k0 + r * kWave + lane, a.n_old - 1);
    in.id[r] = a.order_old[k];
    in.w0[r] = (uint64_t)a.wait_old[k];
  }
  const int64_t j = (int64_t)(uint32_t)d + lane;
  const int64_t jc = min(j, max(a.m - 1, (int64_t)0));  // ins / wait_m hold >= 1 entry
  in.sins = a.ins[jc];
  const uint64_t wm = (uint64_t)a.wait_m[jc];
  in.spn = j < a.m ? wm : lnew;
}

// Entries k0 .. k1-1 of the earlier schedule, c0 = c(k0), ns = arrivals
// inside the unit. Lane handles k = k0 + r * 64 + lane in round r.
// WIDE (ns >= 64): each lane searches the unit's arrivals in global memory.
// Else the unit's arrivals are in the lanes of in.sins / in.spn: a uniform
// pointer p counts those below the round's first entry and only the few in
// the round's 64 positions are compared per lane.
// MIXED: the unit spans several classes; a lane's class is looked up per
// round (else every entry is in class cls0 and `cur` already holds it).
template <bool MIXED, bool WIDE>
__device__ __forceinline__ void merge_unit(const InsArgs& a, const MergeShared& sh,
                                           MergeShared& shw, const UnitIn& in, int64_t k0,
                                           int64_t k1, int64_t c0, int ns, int cls0, int clsL,
                                           int lane, uint64_t lnew, int64_t n, int& cur,
                                           U128& acc) {
  int p = 0;
#pragma unroll
  for (int r = 0; r < MR; ++r) {
    const int64_t kr = k0 + r * kWave;
    const int64_t k = kr + lane;
    int64_t c;
    uint64_t pn;
    if (WIDE) {
      int lo = 0, hi = ns;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (a.ins[c0 + mid] <= (uint32_t)k) lo = mid + 1; else hi = mid;
      }
      c = lo;
      pn = c0 + c < a.m ? (uint64_t)a.wait_m[c0 + c] : lnew;
    } else {
      int q = p, cnt = 0;
      while (q < ns) {
        const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)in.sins, q);
        if (v > (uint32_t)(kr + kWave - 1)) break;
        cnt += v <= (uint32_t)k ? 1 : 0;
        ++q;
      }
      c = p + cnt;
      pn = q == p ? readlane64(in.spn, p) : bpermute64(in.spn, (int)c);
      p = q;
    }
    const uint64_t wt = in.w0[r] + pn;
    const int64_t dst = k + c0 + c;
    const bool live = k < k1;
    const bool ok = live && dst < n;  // (dst < n always, for a consistent earlier schedule)
    int32_t* po = ok ? a.order + dst : reinterpret_cast<int32_t*>(a.sink);
    int64_t* pw = ok ? a.wait + dst : reinterpret_cast<int64_t*>(a.sink + 1);
    *po = in.id[r];
    *pw = (int64_t)wt;
    if (MIXED) {
      int cls = cls0;
      for (int cc = cls0 + 1; cc <= clsL; ++cc) cls += sh.cs[cc] <= (uint32_t)k ? 1 : 0;
      if (cls != cur) {
        flush(shw, cur, acc);
        cur = cls;
      }
    }
    add128(acc, live ? wt : 0);
  }
}

// A wave walks units w, w + waves, ... of the earlier schedule, loading the
// next unit before storing the current one, then places arrivals 64 at a time.
// Per-lane class sums go to LDS when a lane's class changes, LDS to the global
// totals once per block.
__global__ __launch_bounds__(MT) void i_merge(InsArgs a, int64_t units) {
  __shared__ MergeShared sh;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  sh.clo[t] = sh.chi[t] = 0;
  for (int c = t; c < kClassSlots; c += MT) sh.cs[c] = a.cs[c];
  block_sync();
  const int64_t waves = (int64_t)gridDim.x * (MT / kWave);
  const int64_t w =
      (int64_t)blockIdx.x * (MT / kWave) + __builtin_amdgcn_readfirstlane(t / kWave);
  const int64_t n = a.n_old + a.m;
  const uint64_t lnew = a.lsum[1], lold = a.lsum[0];
  ConstU64* desc = (ConstU64*)a.desc;  // address-space cast
  int cur = -1;
  U128 acc = {0, 0};
  if (w < units) {
    int64_t u = w;
    uint64_t d0 = desc[u], d1 = desc[u + 1];
    UnitIn in;
    load_unit(a, u, d0, lane, lnew, in);
    for (;;) {
      const int64_t un = u + waves;
      const bool more = un < units;
      const int64_t uu = more ? un : u;
      const uint64_t e0 = desc[uu], e1 = desc[uu + 1];
      UnitIn nx;
      load_unit(a, uu, e0, lane, lnew, nx);
      const int64_t k0 = u * kInsUnit, k1 = min(a.n_old, k0 + kInsUnit);
      const int64_t c0 = (int64_t)(uint32_t)d0;
      const int64_t c1 = (int64_t)(uint32_t)d1;
      const int ns = c1 > c0 ? (int)(c1 - c0) : 0;
      const int cls0 = (int)(d0 >> 32) & 255, clsL = (int)(d0 >> 40) & 255;
      if (ns >= kWave) {
        merge_unit<true, true>(a, sh, sh, in, k0, k1, c0, ns, cls0, clsL, lane, lnew, n, cur, acc);
      } else if (cls0 != clsL) {
        merge_unit<true, false>(a, sh, sh, in, k0, k1, c0, ns, cls0, clsL, lane, lnew, n, cur,
                                acc);
      } else {
        if (cur != cls0) {
          flush(sh, cur, acc);
          cur = cls0;
        }
        merge_unit<false, false>(a, sh, sh, in, k0, k1, c0, ns, cls0, clsL, lane, lnew, n, cur,
                                 acc);
      }
      if (!more) break;
      u = un;
      d0 = e0;
      d1 = e1;
      in = nx;
    }
  }
  for (int64_t j0 = w * kWave; j0 < a.m; j0 += waves * kWave) {
    const int64_t j = j0 + lane;
    const bool live = j < a.m;
    const int64_t jc = min(j, a.m - 1);
    const int64_t id = a.n_old + clamp_id(a.order_m[jc], a.m);
    const uint64_t wn = (uint64_t)a.wait_m[jc];
    const int64_t at = min((int64_t)a.ins[jc], a.n_old);
    const uint64_t wt = wn + (at < a.n_old ? (uint64_t)a.wait_old[at] : lold);
    const int64_t dst = at + j;
    if (live && dst < n) {
      a.order[dst] = (int32_t)id;
      a.wait[dst] = (int64_t)wt;
    }
    if (live) {
      const int cls = a.priority[id];
      if (cls != cur) {
        flush(sh, cur, acc);
        cur = cls;
      }
      add128(acc, wt);
    }
  }
  flush(sh, cur, acc);
  block_sync();
  const U128 v = {sh.clo[t], sh.chi[t]};  // class t
  if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + t), a.totals + 2 * (1 + t) + 1, v);
  const U128 s = wave_sum128(v);
  if (lane == 0) sh.wsum[t / kWave] = s;
  block_sync();
  if (t == 0) {
    U128 g = {0, 0};
    for (int i = 0; i < MT / kWave; ++i) add128(g, sh.wsum[i]);
    if (g.lo | g.hi) atomic_add128(a.totals, a.totals + 1, g);
  }
}

int merge_resident_blocks() {
  int dev = 0, cus = 256, occ = 1;
  if (hipGetDevice(&dev) == hipSuccess) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) cus = prop.multiProcessorCount;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, reinterpret_cast<const void*>(i_merge),
                                                   MT, 0) != hipSuccess ||
      occ < 1)
    occ = 1;
  return cus * occ;
}

}  // namespace

int64_t insert_units(int64_t n_old) { return (n_old + kInsUnit - 1) / kInsUnit; }

hipError_t launch_insert(const InsArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after) {
  const int64_t units = insert_units(a.n_old);
  const int64_t searches = a.m + units + 1 + kClassSlots + 1;
  hipLaunchKernelGGL(i_search, dim3((unsigned)((searches + IT - 1) / IT)), dim3(IT), 0, st, a,
                     units);
  static const int resident = merge_resident_blocks();
  const int64_t work = std::max(units, (a.m + kWave - 1) / kWave);  // in waves
  int64_t grid = (work + MT / kWave - 1) / (MT / kWave);
  grid = std::min<int64_t>(grid, std::min<int64_t>(resident, kMaxMergeBlocks));
  if (before) (void)hipEventRecord(before, st);
  if (grid > 0) hipLaunchKernelGGL(i_merge, dim3((unsigned)grid), dim3(MT), 0, st, a, units);
  if (after) (void)hipEventRecord(after, st);
  return hipGetLastError();
}

}  // namespace semsched
