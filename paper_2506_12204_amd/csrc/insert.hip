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
#include <algorithm>

#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int IT = 256;          // threads of the insertion kernels
constexpr int IK = 16;           // rounds: a block merges IT * IK entries
constexpr int ITILE = IT * IK;
constexpr int kClassSlots = 257;  // class starts per sequence (classes 0..255 and the end)
constexpr int64_t kMergeBlocks = 2048;  // workgroups of the merge pass (tiles are walked)

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

constexpr int kSliceCap = 256;  // arrivals inside one tile held in LDS (more: searched in global)
constexpr int kCountCap = 32;   // up to this many, every lane counts them all (no search)

struct MergeShared {
  uint32_t cs[kClassSlots];   // class starts of this block's sequence
  uint64_t clo[256], chi[256];
  int64_t cbase[2];           // c(k) at the first and at the last entry of the tile
  int32_t ncb, cls0;          // class starts inside the tile; the class at its first entry
  uint32_t cb[kClassSlots];   // those class starts
  uint32_t slice[kSliceCap];  // insertion points of the arrivals landing inside the tile
  uint64_t pnew[kSliceCap + 1];  // length prefix of the arrivals at c(k0) .. c(k1 - 1)
};

// Number of the first `count` entries of a non-decreasing LDS table that are
// <= x: with few entries every lane counts them all (broadcast reads, a
// uniform trip count), else a binary search.
__device__ __forceinline__ int count_le(const uint32_t* table, int count, uint32_t x) {
  if (count <= kCountCap) {
    int c = 0;
    for (int i = 0; i < count; ++i) c += table[i] <= x ? 1 : 0;
    return c;
  }
  int lo = 0, hi = count;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (table[mid] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Tiles 0 .. old_tiles-1 move earlier entries; the rest place arrivals. A
// block walks tiles blockIdx.x, blockIdx.x + gridDim.x, ... and adds its
// class totals to the global ones once, at the end (a grid of a few
// thousand blocks keeps those 128-bit atomics on a dozen words rare).
// Within a tile a lane handles entries k0 + r * IT + lane (r = 0 .. IK-1):
// consecutive lanes read and write consecutive entries, and a lane's
// entries increase, so its class only moves forward.
__global__ __launch_bounds__(IT) void i_merge(InsArgs a, int64_t old_tiles, int64_t tiles) {
  __shared__ MergeShared sh;
  const int t = threadIdx.x;
  for (int c = t; c < 256; c += IT) sh.clo[c] = sh.chi[c] = 0;
  const uint64_t lnew = a.lsum[1], lold = a.lsum[0];
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const bool arrivals = tile >= old_tiles;
    const int64_t cnt = arrivals ? a.m : a.n_old;  // entries of this tile's sequence
    const int64_t k0 = (arrivals ? tile - old_tiles : tile) * ITILE;
    const int64_t k1 = min(cnt, k0 + ITILE);       // (k0 < k1 for every tile)
    block_sync();  // the previous tile's tables are no longer read
    for (int c = t; c < kClassSlots; c += IT) sh.cs[c] = a.cs[(arrivals ? kClassSlots : 0) + c];
    if (!arrivals && t < 2) {
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
    if (t == 0) {
      // the class of the tile's first entry and the class starts inside the tile
      const int c0 = last_le(sh.cs, 0, 256, (uint32_t)k0);
      int nc = 0;
      for (int c = c0 + 1; c < 256 && sh.cs[c] < (uint32_t)k1; ++c) sh.cb[nc++] = sh.cs[c];
      sh.cls0 = c0;
      sh.ncb = nc;
    }
    const int64_t c0 = arrivals ? 0 : sh.cbase[0];
    const int64_t ns = arrivals ? 0 : sh.cbase[1] - c0;  // arrivals landing inside the tile
    const bool in_lds = ns <= kSliceCap;
    if (!arrivals && in_lds) {
      for (int64_t i = t; i < ns; i += IT) sh.slice[i] = a.ins[c0 + i];
      for (int64_t i = t; i <= ns; i += IT)
        sh.pnew[i] = c0 + i < a.m ? (uint64_t)a.wait_m[c0 + i] : lnew;
    }
    block_sync();
    const int ncb = sh.ncb, cls0 = sh.cls0;

    // every round's inputs first, so that their loads overlap
    int32_t id[IK];
    uint64_t w0[IK];
    uint32_t at[IK];
#pragma unroll
    for (int r = 0; r < IK; ++r) {
      const int64_t k = min(k0 + (int64_t)r * IT + t, k1 - 1);
      if (!arrivals) {
        id[r] = a.order_old[k];
        w0[r] = (uint64_t)a.wait_old[k];
      } else {
        id[r] = (int32_t)(a.n_old + a.order_m[k]);
        w0[r] = (uint64_t)a.wait_m[k];
        at[r] = (uint32_t)min((int64_t)a.ins[k], a.n_old);
      }
    }
    int cur = -1;  // this lane's current class and its 128-bit wait sum
    U128 acc = {0, 0};
#pragma unroll
    for (int r = 0; r < IK; ++r) {
      const int64_t k = k0 + (int64_t)r * IT + t;
      int64_t q;
      uint64_t wt;
      if (!arrivals) {
        // arrivals ahead of earlier entry k: c0 + those of the tile's slice at or before k
        int64_t c;
        uint64_t pn;
        if (in_lds) {
          c = count_le(sh.slice, (int)ns, (uint32_t)k);
          pn = sh.pnew[c];
        } else {
          int64_t lo = 0, hi = ns;
          while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (a.ins[c0 + mid] <= (uint32_t)k) lo = mid + 1; else hi = mid;
          }
          c = lo;
          pn = c0 + c < a.m ? (uint64_t)a.wait_m[c0 + c] : lnew;
        }
        q = k + c0 + c;
        wt = w0[r] + pn;
      } else {
        q = (int64_t)at[r] + k;
        wt = w0[r] + (at[r] < a.n_old ? (uint64_t)a.wait_old[at[r]] : lold);
      }
      if (k < k1 && q < a.n_old + a.m) {  // (q < n always, for a consistent earlier schedule)
        a.order[q] = id[r];
        a.wait[q] = (int64_t)wt;
      }
      if (k < k1) {
        const int cls = cls0 + count_le(sh.cb, ncb, (uint32_t)k);
        if (cls != cur) {
          if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
          cur = cls;
          acc = {0, 0};
        }
        add128(acc, wt);
      }
    }
    if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
  }
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

hipError_t launch_insert(const InsArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after) {
  const int64_t searches = a.m + 2 * kClassSlots + 1;
  hipLaunchKernelGGL(i_search, dim3((unsigned)((searches + IT - 1) / IT)), dim3(IT), 0, st, a);
  const int64_t old_tiles = (a.n_old + ITILE - 1) / ITILE;
  const int64_t tiles = old_tiles + (a.m + ITILE - 1) / ITILE;
  const int64_t grid = std::min<int64_t>(tiles, kMergeBlocks);
  if (before) (void)hipEventRecord(before, st);
  if (grid > 0)
    hipLaunchKernelGGL(i_merge, dim3((unsigned)grid), dim3(IT), 0, st, a, old_tiles, tiles);
  if (after) (void)hipEventRecord(after, st);
  return hipGetLastError();
}

}  // namespace semsched
