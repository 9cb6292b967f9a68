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
//             by binary search over order_old; the class starts of both
//             sequences; the total length of each.
//   i_merge   earlier entry k moves to k + c(k), c(k) = the number of
//             arrivals with ins[j] <= k, and its wait grows by the lengths of
//             those c(k) arrivals (their prefix sum); arrival j lands at
//             ins[j] + j with wait = (earlier wait at ins[j]) + (its wait
//             among the arrivals). Class totals are summed on the way (the
//             merged schedule is class-major, as both inputs are).
//
// Only the arrivals are sorted; every earlier entry is read and written
// once (4 + 8 bytes each way).
#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int IT = 256;          // threads of the insertion kernels
constexpr int IK = 16;           // rounds: a block merges IT * IK entries
constexpr int ITILE = IT * IK;
constexpr int kClassSlots = 257;  // class starts per sequence (classes 0..255 and the end)

// key of an earlier entry / of an arrival, both as (priority, length)
struct KeyPL {
  uint32_t p, l;
};

__device__ __forceinline__ bool key_le(KeyPL a, KeyPL b) {
  return a.p < b.p || (a.p == b.p && a.l <= b.l);
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

// Threads 0 .. m-1: ins[j]. Threads m .. m+256: class start c of the earlier
// sequence (the number of its entries with priority < c); the next 257:
// class starts of the arrivals; one more: the two length totals.
__global__ __launch_bounds__(IT) void i_search(InsArgs a) {
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
  const int64_t r = i - a.m;
  if (r < 2 * kClassSlots) {
    const bool arrivals = r >= kClassSlots;
    const uint32_t c = (uint32_t)(arrivals ? r - kClassSlots : r);
    int64_t lo = 0, hi = arrivals ? a.m : a.n_old;  // first entry with priority >= c
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      const uint32_t pm = arrivals ? new_key(a, mid).p : old_key(a, mid).p;
      if (pm < c) lo = mid + 1; else hi = mid;
    }
    a.cs[r] = (uint32_t)lo;
    return;
  }
  if (r == 2 * kClassSlots) {
    // total lengths: last wait + last length of each sequence
    a.lsum[0] = a.n_old > 0 ? (uint64_t)a.wait_old[a.n_old - 1] + old_key(a, a.n_old - 1).l : 0;
    a.lsum[1] = a.m > 0 ? (uint64_t)a.wait_m[a.m - 1] + new_key(a, a.m - 1).l : 0;
  }
}

// Last index c in [lo, hi] with table[c] <= x, given table[lo] <= x (the
// tables are non-decreasing; equal starts are empty classes, and the last
// one is the class that holds x).
__device__ __forceinline__ int last_le(const uint32_t* table, int lo, int hi, uint32_t x) {
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (table[mid] <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

struct MergeShared {
  uint32_t cs[kClassSlots];   // class starts of this block's sequence
  uint64_t clo[256], chi[256];
  int64_t cbase[2];           // c(k) at the first and last entry of the tile
};

// Blocks 0 .. old_blocks-1 move earlier entries; the rest place arrivals.
__global__ __launch_bounds__(IT) void i_merge(InsArgs a, int64_t old_blocks) {
  __shared__ MergeShared sh;
  const int t = threadIdx.x;
  const bool arrivals = (int64_t)blockIdx.x >= old_blocks;
  const int64_t blk = arrivals ? (int64_t)blockIdx.x - old_blocks : (int64_t)blockIdx.x;
  const int64_t cnt = arrivals ? a.m : a.n_old;  // entries of this block's sequence
  const int64_t k0 = blk * ITILE;
  const int64_t k1 = min(cnt, k0 + ITILE);
  for (int c = t; c < kClassSlots; c += IT) sh.cs[c] = a.cs[(arrivals ? kClassSlots : 0) + c];
  for (int c = t; c < 256; c += IT) sh.clo[c] = sh.chi[c] = 0;
  if (!arrivals && t < 2 && k1 > k0) {
    // c(k) = number of arrivals with ins[j] <= k, at k0 and at k1 - 1
    const uint32_t x = (uint32_t)(t == 0 ? k0 : k1 - 1);
    int64_t lo = 0, hi = a.m;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (a.ins[mid] <= x) lo = mid + 1; else hi = mid;
    }
    sh.cbase[t] = lo;
  }
  block_sync();

  const uint64_t lnew = a.lsum[1], lold = a.lsum[0];
  int cur = -1;          // this lane's current class and its 128-bit wait sum
  U128 acc = {0, 0};
  const int64_t clo_k = arrivals ? 0 : sh.cbase[0];
  const int64_t chi_k = arrivals ? 0 : sh.cbase[1];
  int cls = 0;
  for (int r = 0; r < IK; ++r) {
    const int64_t k = k0 + (int64_t)r * IT + t;
    if (k >= k1) break;
    int64_t q;
    int32_t id;
    uint64_t wt;
    if (!arrivals) {
      // arrivals ahead of earlier entry k: c(k) in [clo_k, chi_k]
      int64_t lo = clo_k, hi = chi_k;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a.ins[mid] <= (uint32_t)k) lo = mid + 1; else hi = mid;
      }
      const int64_t c = lo;
      q = k + c;
      id = a.order_old[k];
      wt = (uint64_t)a.wait_old[k] + (c < a.m ? (uint64_t)a.wait_m[c] : lnew);
    } else {
      const int64_t at = min((int64_t)a.ins[k], a.n_old);
      q = at + k;
      id = (int32_t)(a.n_old + a.order_m[k]);
      wt = (uint64_t)a.wait_m[k] + (at < a.n_old ? (uint64_t)a.wait_old[at] : lold);
    }
    if (q < a.n_old + a.m) {  // always true for a consistent earlier schedule
      a.order[q] = id;
      a.wait[q] = (int64_t)wt;
    }
    cls = last_le(sh.cs, cls, 256, (uint32_t)k);  // classes never decrease along a lane
    if (cls != cur) {
      if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
      cur = cls;
      acc = {0, 0};
    }
    add128(acc, wt);
  }
  if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
  block_sync();
  for (int c = t; c < 256; c += IT) {
    U128 v = {sh.clo[c], sh.chi[c]};
    if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + c), a.totals + 2 * (1 + c) + 1, v);
  }
  if (t == 0) {
    U128 g = {0, 0};
    for (int c = 0; c < 256; ++c) add128(g, U128{sh.clo[c], sh.chi[c]});
    if (g.lo | g.hi) atomic_add128(a.totals, a.totals + 1, g);
  }
}

}  // namespace

hipError_t launch_insert(const InsArgs& a, hipStream_t st) {
  const int64_t searches = a.m + 2 * kClassSlots + 1;
  hipLaunchKernelGGL(i_search, dim3((unsigned)((searches + IT - 1) / IT)), dim3(IT), 0, st, a);
  const int64_t old_blocks = (a.n_old + ITILE - 1) / ITILE;
  const int64_t new_blocks = (a.m + ITILE - 1) / ITILE;
  if (old_blocks + new_blocks > 0)
    hipLaunchKernelGGL(i_merge, dim3((unsigned)(old_blocks + new_blocks)), dim3(IT), 0, st, a,
                       old_blocks);
  return hipGetLastError();
}

}  // namespace semsched
