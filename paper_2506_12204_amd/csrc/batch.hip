// Batch selection with stage awareness (Algorithm 2) and priority-based
// eviction (Algorithms 3 and 4) of Section 3.3.
//
// Both work on the few requests of one scheduling iteration (candidates,
// ongoing requests, cached requests), so each is one workgroup over LDS.
// A request's key is (rank << 32 | length, id): the scheduling order of
// Algorithm 1; the smallest key is the most urgent request.
//
//   b_select  sorts the candidates (the heap's first b entries and the
//             unsorted buffer) and the ongoing requests with a bitonic
//             network; the candidates C are the first b. The most urgent of
//             C and O decides the stage filter; every element's place in
//             the merged list M (C's surviving members and O) and in the
//             pushed-back list (C's filtered members and M beyond b) comes
//             from binary searches in the other sorted lists.
//   b_evict   sorts the cached requests; the eviction order is that order
//             reversed (least urgent, longest first; the later arrival
//             first among equal keys). A scan of their KV sizes in that
//             order gives, for each incoming request, the number of
//             victims after its step: the shortest prefix covering
//             usage + (demands so far) - capacity.
#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int BT = 1024;
constexpr int kCandCap = 2 * kSelectCap;  // heap's first b plus the buffer

__device__ __forceinline__ bool less(uint64_t ka, uint32_t ia, uint64_t kb, uint32_t ib) {
  return ka < kb || (ka == kb && ia < ib);
}

// The value of lane (this lane ^ M). Distances 1, 2 and 8 are one DPP move
// (quad permutes; a rotation of the 16-lane row by 8), 4 is two row shifts
// and a select: no LDS traffic. 16 and 32 cross rows: a bpermute.
template <int M>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v) {
  if constexpr (M == 1) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xb1, 0xf, 0xf, false);  // quad_perm [1,0,3,2]
  } else if constexpr (M == 2) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4e, 0xf, 0xf, false);  // quad_perm [2,3,0,1]
  } else if constexpr (M == 4) {
    const uint32_t up = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x104, 0xf, 0xf, false);
    const uint32_t dn = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);
    return (lane_id() & 4) ? dn : up;  // row_shl:4 (lane + 4), row_shr:4 (lane - 4)
  } else if constexpr (M == 8) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xf, 0xf, false);  // row_ror:8
  } else {
    return (uint32_t)__shfl_xor((int)v, M, kWave);
  }
}

template <int M>
__device__ __forceinline__ uint64_t xor_lane64(uint64_t v) {
  return (uint64_t)xor_lane<M>((uint32_t)(v >> 32)) << 32 | xor_lane<M>((uint32_t)v);
}

// Ascending bitonic sort of BT * E (key, id) pairs in LDS, with an optional
// u32 payload that moves with them. Thread t holds elements t*E .. t*E+E-1 in
// registers throughout: compare-exchange distances below E stay inside a
// thread, distances below 64 * E pair a lane with another lane of its wave
// (shuffles, no barrier), and only the longer ones go through LDS with
// workgroup barriers. Every thread of the block must call it.
template <int E, bool PAYLOAD>
__device__ void block_sort(uint64_t* key, uint32_t* id, uint32_t* pay) {
  constexpr uint32_t N = BT * E;
  const uint32_t t = threadIdx.x, lane = t & (kWave - 1);
  uint64_t xk[E];
  uint32_t xi[E], xp[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    xk[e] = key[t * E + e];
    xi[e] = id[t * E + e];
    xp[e] = PAYLOAD ? pay[t * E + e] : 0u;
  }
  // element (t*E + e) meets its partner; keep the smaller when take_min
  auto keep = [&](int e, bool take_min, uint64_t pk, uint32_t pi, uint32_t pp) {
    const bool pless = less(pk, pi, xk[e], xi[e]);
    if (take_min == pless) {
      xk[e] = pk;
      xi[e] = pi;
      xp[e] = pp;
    }
  };
  for (uint32_t k = 2; k <= N; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      if (j < (uint32_t)E) {
#pragma unroll
        for (int jj = E / 2; jj >= 1; jj >>= 1) {
          if (j != (uint32_t)jj) continue;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            if (e & jj) continue;
            const int f = e | jj;
            const bool up = ((t * E + e) & k) == 0;
            if (less(xk[f], xi[f], xk[e], xi[e]) == up) {
              const uint64_t tk = xk[e];
              const uint32_t ti = xi[e], tp = xp[e];
              xk[e] = xk[f];
              xi[e] = xi[f];
              xp[e] = xp[f];
              xk[f] = tk;
              xi[f] = ti;
              xp[f] = tp;
            }
          }
        }
      } else if (j < (uint32_t)(kWave * E)) {
        const int m = (int)(j / E);  // partner lane = lane ^ m
        const bool take_min = ((lane & m) == 0) == (((t * E) & k) == 0);
        auto stage = [&](auto mc) {
          constexpr int M = decltype(mc)::value;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const uint64_t pk = xor_lane64<M>(xk[e]);
            const uint32_t pi = xor_lane<M>(xi[e]);
            const uint32_t pp = PAYLOAD ? xor_lane<M>(xp[e]) : 0u;
            keep(e, take_min, pk, pi, pp);
          }
        };
        switch (m) {  // (uniform)
          case 1: stage(std::integral_constant<int, 1>{}); break;
          case 2: stage(std::integral_constant<int, 2>{}); break;
          case 4: stage(std::integral_constant<int, 4>{}); break;
          case 8: stage(std::integral_constant<int, 8>{}); break;
          case 16: stage(std::integral_constant<int, 16>{}); break;
          default: stage(std::integral_constant<int, 32>{}); break;
        }
      } else {
        const uint32_t m = j / E;  // partner thread = t ^ m, another wave
        const bool take_min = ((t & m) == 0) == (((t * E) & k) == 0);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          key[t * E + e] = xk[e];
          id[t * E + e] = xi[e];
          if (PAYLOAD) pay[t * E + e] = xp[e];
        }
        block_sync();
        const uint32_t pt = t ^ m;
#pragma unroll
        for (int e = 0; e < E; ++e)
          keep(e, take_min, key[pt * E + e], id[pt * E + e], PAYLOAD ? pay[pt * E + e] : 0u);
        block_sync();
      }
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    key[t * E + e] = xk[e];
    id[t * E + e] = xi[e];
    if (PAYLOAD) pay[t * E + e] = xp[e];
  }
  block_sync();
}

// Sorts the first n entries (n <= 8 * BT; entries from n up to the sort
// size must hold the sentinel key ~0).
template <bool PAYLOAD>
__device__ void sort_pairs(uint64_t* key, uint32_t* id, uint32_t* pay, uint32_t n) {
  if (n <= (uint32_t)BT) block_sort<1, PAYLOAD>(key, id, pay);
  else if (n <= 2u * BT) block_sort<2, PAYLOAD>(key, id, pay);
  else if (n <= 4u * BT) block_sort<4, PAYLOAD>(key, id, pay);
  else block_sort<8, PAYLOAD>(key, id, pay);
}

__device__ __forceinline__ uint32_t sort_size(uint32_t n) {
  return n <= (uint32_t)BT ? BT : n <= 2u * BT ? 2 * BT : n <= 4u * BT ? 4 * BT : 8 * BT;
}

// Number of entries of a sorted list below (k, i).
__device__ __forceinline__ uint32_t count_below(const uint64_t* key, const uint32_t* id,
                                                uint32_t n, uint64_t k, uint32_t i) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (less(key[mid], id[mid], k, i)) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ uint64_t key_of(const SelArgs& a, uint32_t id) {
  return (uint64_t)a.priority[id] << 32 | (uint32_t)a.length[id];
}

struct SelectShared {
  uint64_t ckey[kCandCap];
  uint32_t cid[kCandCap];
  uint64_t okey[kSelectCap];
  uint32_t oid[kSelectCap];
  uint16_t dec_excl[kSelectCap + 1];  // kept members of C before each index (<= 4096)
  uint32_t scan32[BT / kWave + 1];
  uint32_t bad;
};

__global__ __launch_bounds__(BT) void b_select(SelArgs a) {
  __shared__ SelectShared sh;
  const uint32_t t = threadIdx.x;
  const uint32_t nh = (uint32_t)min(a.b, a.n_heap);
  const uint32_t nc_in = nh + (uint32_t)a.n_buffer;
  const uint32_t no = (uint32_t)a.n_ongoing;
  const uint32_t NC = sort_size(nc_in), NO = sort_size(no);
  if (t == 0) sh.bad = 0;
  block_sync();
  // gather the keys; ids outside [0, n_ids) are reported and sort last
  for (uint32_t i = t; i < NC; i += BT) {
    uint64_t k = ~0ull;
    uint32_t id = ~0u;
    if (i < nc_in) {
      const int32_t v = i < nh ? a.heap_order[i] : a.buffer[i - nh];
      if (v >= 0 && v < a.n_ids) {
        id = (uint32_t)v;
        k = key_of(a, id);
      } else {
        atomicOr(&sh.bad, 1u);
      }
    }
    sh.ckey[i] = k;
    sh.cid[i] = id;
  }
  for (uint32_t i = t; i < NO; i += BT) {
    uint64_t k = ~0ull;
    uint32_t id = ~0u;
    if (i < no) {
      const int32_t v = a.ongoing[i];
      if (v >= 0 && v < a.n_ids) {
        id = (uint32_t)v;
        k = key_of(a, id);
      } else {
        atomicOr(&sh.bad, 1u);
      }
    }
    sh.okey[i] = k;
    sh.oid[i] = id;
  }
  block_sync();
  if (sh.bad) {
    if (t == 0) {
      atomicOr(a.flags, kFlagInval);
      a.counts[0] = a.counts[1] = 0;
    }
    return;
  }
  sort_pairs<false>(sh.ckey, sh.cid, nullptr, nc_in);
  sort_pairs<false>(sh.okey, sh.oid, nullptr, no);
  const uint32_t nc = min((uint32_t)a.b, nc_in);  // C = the first nc candidates
  if (nc == 0 && no == 0) {
    if (t == 0) a.counts[0] = a.counts[1] = 0;
    return;
  }
  // the most urgent of C and O decides whether prefill candidates stay
  bool top_in_c = nc > 0 && (no == 0 || less(sh.ckey[0], sh.cid[0], sh.okey[0], sh.oid[0]));
  const uint32_t top = top_in_c ? sh.cid[0] : sh.oid[0];
  const bool keep_all = a.stage[top] == 0;
  // decoding (kept) members of C before each index: each thread scans a
  // chunk of consecutive candidates
  constexpr uint32_t PER = (kSelectCap + BT - 1) / BT;
  const uint32_t c0 = min(nc, t * PER), c1 = min(nc, c0 + PER);
  uint32_t mine = 0;
  for (uint32_t i = c0; i < c1; ++i) mine += (keep_all || a.stage[sh.cid[i]] != 0) ? 1u : 0u;
  uint32_t ndec;
  uint32_t run = block_excl_scan_u32<BT>(mine, sh.scan32, ndec);
  for (uint32_t i = c0; i < c1; ++i) {
    sh.dec_excl[i] = (uint16_t)run;
    run += (keep_all || a.stage[sh.cid[i]] != 0) ? 1u : 0u;
  }
  if (t == 0) sh.dec_excl[nc] = (uint16_t)ndec;
  block_sync();
  const uint32_t nm = ndec + no;           // |M|
  const uint32_t b = (uint32_t)a.b;
  const uint32_t npre = nc - ndec;
  const uint32_t over = nm > b ? nm - b : 0;  // M beyond the batch
  // members of M below (k, i): kept members of C and members of O
  auto m_below = [&](uint64_t k, uint32_t i) {
    const uint32_t c = count_below(sh.ckey, sh.cid, nc, k, i);
    return sh.dec_excl[c] + count_below(sh.okey, sh.oid, no, k, i);
  };
  // filtered (prefill) members of C below (k, i)
  auto pre_below = [&](uint64_t k, uint32_t i) {
    const uint32_t c = count_below(sh.ckey, sh.cid, nc, k, i);
    return c - sh.dec_excl[c];
  };
  auto place_m = [&](uint32_t q, uint32_t id, uint64_t k) {  // q = position in M
    if (q < b) {
      a.batch[q] = (int32_t)id;
    } else {
      a.pushed[(q - b) + pre_below(k, id)] = (int32_t)id;
    }
  };
  for (uint32_t i = t; i < nc; i += BT) {
    const uint64_t k = sh.ckey[i];
    const uint32_t id = sh.cid[i];
    const uint32_t rk = sh.dec_excl[i];
    const bool kept = (uint32_t)sh.dec_excl[i + 1] != rk;
    if (kept) {
      place_m(rk + count_below(sh.okey, sh.oid, no, k, id), id, k);
    } else {
      const uint32_t mb = m_below(k, id);
      a.pushed[(i - rk) + (mb > b ? mb - b : 0)] = (int32_t)id;
    }
  }
  for (uint32_t j = t; j < no; j += BT) {
    const uint64_t k = sh.okey[j];
    const uint32_t id = sh.oid[j];
    place_m(j + sh.dec_excl[count_below(sh.ckey, sh.cid, nc, k, id)], id, k);
  }
  if (t == 0) {
    a.counts[0] = min(b, nm);
    a.counts[1] = npre + over;
  }
}

struct EvictShared {
  uint64_t key[kEvictCap];
  uint32_t id[kEvictCap];
  uint32_t src[kEvictCap];    // index into the caller's cached / kv arrays
  uint64_t scan64[BT / kWave + 1];
  uint32_t bad;
};

__global__ __launch_bounds__(BT) void b_evict(EvictArgs a) {
  __shared__ EvictShared sh;
  const uint32_t t = threadIdx.x;
  const uint32_t nr = (uint32_t)a.n_cached;
  const uint32_t N = sort_size(nr);
  if (t == 0) sh.bad = 0;
  block_sync();
  for (uint32_t i = t; i < N; i += BT) {
    uint64_t k = ~0ull;
    uint32_t id = ~0u;
    if (i < nr) {
      const int32_t v = a.cached[i];
      if (v >= 0 && v < a.n_ids && a.kv[i] >= 0) {
        id = (uint32_t)v;
        k = (uint64_t)a.priority[id] << 32 | (uint32_t)a.length[id];
      } else {
        atomicOr(&sh.bad, v >= 0 && v < a.n_ids ? 2u : 1u);  // 2: negative KV size
      }
    }
    sh.key[i] = k;
    sh.id[i] = id;
    sh.src[i] = i;
  }
  block_sync();
  if (sh.bad) {
    if (t == 0) atomicOr(a.flags, (sh.bad & 1u) ? kFlagInval : kFlagRange);
    return;
  }
  sort_pairs<true>(sh.key, sh.id, sh.src, nr);
  // KV sizes in eviction order (the sorted order read backwards), inclusive
  // prefix sums over a contiguous chunk per thread, kept in sh.key
  constexpr uint32_t PER = (kEvictCap + BT - 1) / BT;
  const uint32_t e0 = min(nr, t * PER), e1 = min(nr, e0 + PER);
  uint64_t kvs[PER];
  uint64_t mine = 0;
#pragma unroll
  for (uint32_t u = 0; u < PER; ++u) {
    const uint32_t e = e0 + u;
    kvs[u] = e < e1 ? (uint64_t)a.kv[sh.src[nr - 1 - e]] : 0;
    mine += kvs[u];
  }
  uint32_t ids[PER];
#pragma unroll
  for (uint32_t u = 0; u < PER; ++u) ids[u] = e0 + u < e1 ? sh.id[nr - 1 - (e0 + u)] : 0;
  uint64_t total;
  uint64_t run = block_excl_scan_u64<BT>(mine, sh.scan64, total);  // (ends with a barrier)
#pragma unroll
  for (uint32_t u = 0; u < PER; ++u) {
    if (e0 + u < e1) {
      run += kvs[u];
      sh.key[e0 + u] = run;      // KV evicted by the first e0+u+1 victims
      sh.id[e0 + u] = ids[u];    // the eviction order
    }
  }
  block_sync();
  // victims after each incoming request j: the first k whose prefix reaches
  // need_j = usage + (demands 0..j) - capacity
  uint32_t k_last = 0;
  bool bad = false;
  int64_t carry = 0;  // demands of the earlier chunks
  for (int64_t j0 = 0; j0 < a.n_demands; j0 += BT) {
    const int64_t j = j0 + t;
    const int64_t s = j < a.n_demands ? a.demands[j] : 0;
    bad |= s < 0;
    uint64_t tot;
    const uint64_t before = block_excl_scan_u64<BT>(s < 0 ? 0 : (uint64_t)s, sh.scan64, tot);
    const int64_t need = a.usage + carry + (int64_t)before + (s < 0 ? 0 : s) - a.capacity;
    uint32_t k = 0;
    if (need > 0) {
      uint32_t lo = 0, hi = nr;  // first index whose inclusive sum reaches need
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if ((int64_t)sh.key[mid] >= need) hi = mid; else lo = mid + 1;
      }
      k = lo < nr ? lo + 1 : nr;
    }
    if (j < a.n_demands) a.upto[j] = k;
    if (j == a.n_demands - 1) sh.bad = k;
    carry += (int64_t)tot;  // (every thread holds the chunk's total)
    block_sync();
  }
  if (__ballot(bad) && lane_id() == 0) atomicOr(a.flags, kFlagRange);
  k_last = a.n_demands > 0 ? sh.bad : 0;
  for (uint32_t e = t; e < k_last; e += BT) a.victims[e] = (int32_t)sh.id[e];
}

}  // namespace

hipError_t launch_select(const SelArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(b_select, dim3(1), dim3(BT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_evict_victims(const EvictArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(b_evict, dim3(1), dim3(BT), 0, st, a);
  return hipGetLastError();
}

}  // namespace semsched
