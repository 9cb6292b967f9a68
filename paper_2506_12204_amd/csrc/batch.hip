// Batch selection with stage awareness (Algorithm 2) and priority-based
// eviction (Algorithms 3 and 4) of Section 3.3.
//
// Both work on the few requests of one scheduling iteration (candidates,
// ongoing requests, cached requests), so each is one workgroup over LDS.
// A request's key is (rank << 32 | length, id): the scheduling order of
// Algorithm 1; the smallest key is the most urgent request.
//
//   b_select  sorts the candidates (the heap's first b entries and the
//             unsorted buffer) and the ongoing requests (an LDS radix sort
//             over the key bits that vary); the candidates C are the first
//             b. The most urgent of C and O decides the stage filter; every
//             element's place in the merged list M (C's surviving members and O) and in the
//             pushed-back list (C's filtered members and M beyond b) comes
//             from binary searches in the other sorted lists.
//   b_evict   sorts the cached requests; the eviction order is that order
//             reversed (least urgent, longest first; the later arrival
//             first among equal keys). A scan of their KV sizes in that
//             order gives, for each incoming request, the number of
//             victims after its step: the shortest prefix covering
//             usage + (demands so far) - capacity.
#include <algorithm>

#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int BT = 1024;
constexpr int kCandCap = 2 * kSelectCap;  // heap's first b plus the buffer

__device__ __forceinline__ bool less(uint64_t ka, uint32_t ia, uint64_t kb, uint32_t ib) {
  return ka < kb || (ka == kb && ia < ib);
}

// Scratch of the block radix sort: per-wave digit counters (then the waves'
// offsets) and the wave partials of the key range reduction and the scans.
constexpr int kSortWaves = BT / kWave;
struct SortScratch {
  uint16_t cnt[kSortWaves][256];
  uint32_t red[kSortWaves * 6];
};

// Stable LSD radix sort by (key, id) of the first n of the BT * E entries of
// key / id (and a u32 payload that moves with them) in LDS, 8 bits at a time,
// the id's digits first, then the key's; digits that are the same for all n
// entries are skipped (the bitwise AND and OR of all keys and ids tell which
// vary). Every pass ranks the rounds of each wave by ballot matching
// (entries (wave, round, lane) in index order, so ranks follow the current
// order: stable), turns the waves' counts into digit-major offsets and
// scatters through LDS. Entries n .. BT*E-1 take (OR of the keys, OR of the
// ids): no real entry sorts after them. Every thread of the block must call
// it.
template <int E, bool PAYLOAD>
__device__ void block_sort(uint64_t* key, uint32_t* id, uint32_t* pay, uint32_t n,
                           SortScratch& sc) {
  if (n <= 1) return;  // (uniform) nothing to order
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  auto at = [&](int r) { return (uint32_t)(w * kWave * E + r * kWave + lane); };
  uint64_t xk[E];
  uint32_t xi[E], xp[E];
  uint32_t kand_lo = ~0u, kand_hi = ~0u, kor_lo = 0, kor_hi = 0, iand = ~0u, ior = 0;
#pragma unroll
  for (int r = 0; r < E; ++r) {
    const uint32_t i = at(r);
    xk[r] = key[i];
    xi[r] = id[i];
    xp[r] = PAYLOAD ? pay[i] : 0u;
    if (i < n) {
      kand_lo &= (uint32_t)xk[r];
      kand_hi &= (uint32_t)(xk[r] >> 32);
      kor_lo |= (uint32_t)xk[r];
      kor_hi |= (uint32_t)(xk[r] >> 32);
      iand &= xi[r];
      ior |= xi[r];
    }
  }
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    kand_lo &= (uint32_t)__shfl_xor((int)kand_lo, off, kWave);
    kand_hi &= (uint32_t)__shfl_xor((int)kand_hi, off, kWave);
    kor_lo |= (uint32_t)__shfl_xor((int)kor_lo, off, kWave);
    kor_hi |= (uint32_t)__shfl_xor((int)kor_hi, off, kWave);
    iand &= (uint32_t)__shfl_xor((int)iand, off, kWave);
    ior |= (uint32_t)__shfl_xor((int)ior, off, kWave);
  }
  if (lane == 0) {
    uint32_t* r6 = sc.red + 6 * w;
    r6[0] = kand_lo, r6[1] = kand_hi, r6[2] = kor_lo, r6[3] = kor_hi, r6[4] = iand, r6[5] = ior;
  }
  block_sync();
#pragma unroll
  for (int v = 0; v < kSortWaves; ++v) {
    const uint32_t* r6 = sc.red + 6 * v;
    kand_lo &= r6[0], kand_hi &= r6[1], kor_lo |= r6[2], kor_hi |= r6[3];
    iand &= r6[4], ior |= r6[5];
  }
  block_sync();  // (the partials' words are the scans' scratch below)
  const uint64_t kor = (uint64_t)kor_hi << 32 | kor_lo;
  uint64_t kvary = kor ^ ((uint64_t)kand_hi << 32 | kand_lo);
  uint32_t ivary = ior ^ iand;
#pragma unroll
  for (int r = 0; r < E; ++r) {
    if (at(r) >= n) {
      xk[r] = kor;
      xi[r] = ior;
    }
  }
  // Packed form: the spans of varying bits of the id, the key's low word and
  // its high word, laid end to end in one u64 (id lowest), when they fit. Its
  // order is the order by (key, id), and its bytes take the passes, in place
  // of the id's and the key's varying bytes (41 bits and 6 passes against 7
  // bytes for ids of 26 bits, lengths of 12 and ranks of 3). The key array
  // then carries the packed value, and the keys are rebuilt from it (and the
  // bits that do not vary) after the last pass.
  const uint32_t v0 = ivary, v1 = (uint32_t)kvary, v2 = (uint32_t)(kvary >> 32);
  const uint32_t l0 = v0 ? __builtin_ctz(v0) : 0, w0 = v0 ? 32 - __builtin_clz(v0) - l0 : 0;
  const uint32_t l1 = v1 ? __builtin_ctz(v1) : 0, w1 = v1 ? 32 - __builtin_clz(v1) - l1 : 0;
  const uint32_t l2 = v2 ? __builtin_ctz(v2) : 0, w2 = v2 ? 32 - __builtin_clz(v2) - l2 : 0;
  const uint32_t pbits = w0 + w1 + w2;
  auto low_mask = [](uint32_t wd) { return wd >= 32 ? ~0u : (1u << wd) - 1u; };
  const uint32_t m0 = low_mask(w0), m1 = low_mask(w1), m2 = low_mask(w2);
  uint32_t vbytes = 0;  // passes of the byte form
#pragma unroll
  for (int b = 0; b < 4; ++b)
    vbytes += ((v0 >> (8 * b)) & 0xffu ? 1u : 0u) + ((v1 >> (8 * b)) & 0xffu ? 1u : 0u) +
              ((v2 >> (8 * b)) & 0xffu ? 1u : 0u);
  const bool packed = pbits <= 64 && (pbits + 7) / 8 < vbytes;
  const uint32_t s2 = w0 + w1;  // below 64 when the high word's span is not empty
  bool packed_moved = false;  // the key array holds packed values
  if (packed) {
#pragma unroll
    for (int r = 0; r < E; ++r) {
      const uint64_t f0 = (xi[r] >> l0) & m0;
      const uint64_t f1 = ((uint32_t)xk[r] >> l1) & m1;
      const uint64_t f2 = ((uint32_t)(xk[r] >> 32) >> l2) & m2;
      xk[r] = f0 | (f1 << w0) | (w2 ? f2 << s2 : 0ull);
    }
    kvary = pbits >= 64 ? ~0ull : (1ull << pbits) - 1;
    ivary = 0;
  }
  uint16_t* mycnt = sc.cnt[w];
  for (int pass = 0; pass < 12; ++pass) {
    const bool on_id = pass < 4;
    const int sh = 8 * (on_id ? pass : pass - 4);
    const uint32_t vary = on_id ? (ivary >> sh) & 0xffu : (uint32_t)(kvary >> sh) & 0xffu;
    if (vary == 0) continue;  // (uniform)
    for (int b = lane; b < 256; b += kWave) mycnt[b] = 0;
    uint32_t dg[E], rk[E];
#pragma unroll
    for (int r = 0; r < E; ++r) {
      dg[r] = on_id ? (xi[r] >> sh) & 0xffu : (uint32_t)(xk[r] >> sh) & 0xffu;
      rk[r] = rank_round_c<8>(dg[r], mycnt);
    }
    block_sync();  // every wave's counts are in
    // digit-major offsets: thread d < 256 owns digit d
    uint32_t c[kSortWaves], tot = 0;
#pragma unroll
    for (int v = 0; v < kSortWaves; ++v) {
      c[v] = t < 256 ? sc.cnt[v][t] : 0u;
      tot += c[v];
    }
    uint32_t all;
    uint32_t run = block_excl_scan_u32<BT>(tot, sc.red, all);
    if (t < 256) {
#pragma unroll
      for (int v = 0; v < kSortWaves; ++v) {
        sc.cnt[v][t] = (uint16_t)run;
        run += c[v];
      }
    }
    block_sync();  // offsets are written
#pragma unroll
    for (int r = 0; r < E; ++r) {
      const uint32_t q = rk[r] + mycnt[dg[r]];
      key[q] = xk[r];
      id[q] = xi[r];
      if (PAYLOAD) pay[q] = xp[r];
    }
    packed_moved = packed;
    block_sync();  // the pass is scattered
#pragma unroll
    for (int r = 0; r < E; ++r) {
      const uint32_t i = at(r);
      xk[r] = key[i];
      xi[r] = id[i];
      if (PAYLOAD) xp[r] = pay[i];
    }
  }
  if (packed_moved) {  // (uniform) the keys back from the packed values
    const uint32_t keep_lo = kand_lo & ~(m1 << l1), keep_hi = kand_hi & ~(m2 << l2);
#pragma unroll
    for (int r = 0; r < E; ++r) {
      const uint32_t f1 = (uint32_t)(xk[r] >> w0) & m1;
      const uint32_t f2 = w2 ? (uint32_t)(xk[r] >> s2) & m2 : 0u;
      key[at(r)] = (uint64_t)(keep_hi | (f2 << l2)) << 32 | (keep_lo | (f1 << l1));
    }
  }
  block_sync();  // (the last pass's reads are done before callers write)
}

// Sorts the first n entries (n <= 8 * BT) of key / id (and pay), with E
// entries per thread, the fewest of 1, 2, 4, 5, 6 or 8 that hold n (each
// pass costs about E rounds per wave, padding included; the sort with a
// payload keeps to 1, 2, 4 and 8, whose kernel the other widths made spill).
template <bool PAYLOAD>
__device__ void sort_pairs(uint64_t* key, uint32_t* id, uint32_t* pay, uint32_t n,
                           SortScratch& sc) {
  if (n <= (uint32_t)BT) block_sort<1, PAYLOAD>(key, id, pay, n, sc);
  else if (n <= 2u * BT) block_sort<2, PAYLOAD>(key, id, pay, n, sc);
  else if (n <= 4u * BT) block_sort<4, PAYLOAD>(key, id, pay, n, sc);
  else if (!PAYLOAD && n <= 5u * BT) block_sort<5, PAYLOAD>(key, id, pay, n, sc);
  else if (!PAYLOAD && n <= 6u * BT) block_sort<6, PAYLOAD>(key, id, pay, n, sc);
  else block_sort<8, PAYLOAD>(key, id, pay, n, sc);
}

template <bool PAYLOAD>
__device__ __forceinline__ uint32_t sort_size(uint32_t n) {
  return n <= (uint32_t)BT ? BT : n <= 2u * BT ? 2 * BT : n <= 4u * BT ? 4 * BT
         : !PAYLOAD && n <= 5u * BT ? 5 * BT : !PAYLOAD && n <= 6u * BT ? 6 * BT : 8 * BT;
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

// Number of entries of a sorted list not above (k, i).
__device__ __forceinline__ uint32_t count_not_above(const uint64_t* key, const uint32_t* id,
                                                    uint32_t n, uint64_t k, uint32_t i) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (!less(k, i, key[mid], id[mid])) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ uint64_t key_of(const SelArgs& a, uint32_t id) {
  return (uint64_t)a.priority[id] << 32 | (uint32_t)a.length[id];
}

// Output of entry idx of C (idx < nc) or of O (idx - nc), given both sorted
// and dec[i] = kept (decoding, or every, when the most urgent entry is in
// prefill) members of C before index i, for i <= nc. M = kept members of C
// and O merged by key; the batch is M's first b; pushed back are C's
// filtered members and M beyond b, merged by key.
template <typename D>
__device__ __forceinline__ void select_place(const SelArgs& a, const uint64_t* ckey,
                                             const uint32_t* cid, uint32_t nc,
                                             const uint64_t* okey, const uint32_t* oid,
                                             uint32_t no, const D* dec, uint32_t idx) {
  // (|M| < 2^31: a larger b places the same way)
  const uint32_t b = (uint32_t)min(a.b, (int64_t)1 << 31);
  // members of M below (k, i): kept members of C and members of O
  auto m_below = [&](uint64_t k, uint32_t i) {
    const uint32_t c = count_below(ckey, cid, nc, k, i);
    return (uint32_t)dec[c] + count_below(okey, oid, no, k, i);
  };
  // filtered (prefill) members of C below (k, i)
  auto pre_below = [&](uint64_t k, uint32_t i) {
    const uint32_t c = count_below(ckey, cid, nc, k, i);
    return c - (uint32_t)dec[c];
  };
  auto place_m = [&](uint32_t q, uint32_t id, uint64_t k) {  // q = position in M
    if (q < b) {
      a.batch[q] = (int32_t)id;
    } else {
      a.pushed[(q - b) + pre_below(k, id)] = (int32_t)id;
    }
  };
  if (idx < nc) {
    const uint32_t i = idx;
    const uint64_t k = ckey[i];
    const uint32_t id = cid[i];
    const uint32_t rk = (uint32_t)dec[i];
    const bool kept = (uint32_t)dec[i + 1] != rk;
    if (kept) {
      place_m(rk + count_below(okey, oid, no, k, id), id, k);
    } else {
      const uint32_t mb = m_below(k, id);
      a.pushed[(i - rk) + (mb > b ? mb - b : 0)] = (int32_t)id;
    }
  } else {
    const uint32_t j = idx - nc;
    const uint64_t k = okey[j];
    const uint32_t id = oid[j];
    place_m(j + (uint32_t)dec[count_below(ckey, cid, nc, k, id)], id, k);
  }
}

struct SelectShared {
  uint64_t ckey[kCandCap];
  uint32_t cid[kCandCap];
  uint64_t okey[kSelectCap];
  uint32_t oid[kSelectCap];
  union {  // (the sorts are done before dec_excl is written)
    uint16_t dec_excl[kSelectCap + 1];  // kept members of C before each index (<= 4096)
    SortScratch sort;
  };
  uint32_t scan32[BT / kWave + 1];
  uint32_t bad;
};

__global__ __launch_bounds__(BT) void b_select(SelArgs a) {
  __shared__ SelectShared sh;
  const uint32_t t = threadIdx.x;
  const uint32_t nh = (uint32_t)min(a.b, a.n_heap);
  const uint32_t nc_in = nh + (uint32_t)a.n_buffer;
  const uint32_t no = (uint32_t)a.n_ongoing;
  const uint32_t NC = sort_size<false>(nc_in), NO = sort_size<false>(no);
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
  sort_pairs<false>(sh.ckey, sh.cid, nullptr, nc_in, sh.sort);
  sort_pairs<false>(sh.okey, sh.oid, nullptr, no, sh.sort);
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
  const uint32_t nm = ndec + no;  // |M|
  const uint32_t b = (uint32_t)a.b;
  const uint32_t npre = nc - ndec;
  const uint32_t over = nm > b ? nm - b : 0;  // M beyond the batch
  for (uint32_t i = t; i < nc + no; i += BT)
    select_place(a, sh.ckey, sh.cid, nc, sh.okey, sh.oid, no, sh.dec_excl, i);
  if (t == 0) {
    a.counts[0] = min(b, nm);
    a.counts[1] = npre + over;
  }
}

// Victims after each incoming request j: the first k of the eviction order
// whose KV prefix psum[k - 1] reaches need_j = usage + (demands 0..j) -
// capacity (all nr if none does); then the victims of the last request, in
// eviction order, from eorder. `last` is a u32 of LDS.
__device__ __forceinline__ void evict_demands(const EvictArgs& a, const uint64_t* psum,
                                              const uint32_t* eorder, uint32_t nr,
                                              uint64_t* scan64, uint32_t* last) {
  const uint32_t t = threadIdx.x;
  bool bad = false;
  int64_t carry = 0;  // demands of the earlier chunks
  for (int64_t j0 = 0; j0 < a.n_demands; j0 += BT) {
    const int64_t j = j0 + t;
    const int64_t s = j < a.n_demands ? a.demands[j] : 0;
    bad |= s < 0;
    uint64_t tot;
    const uint64_t before = block_excl_scan_u64<BT>(s < 0 ? 0 : (uint64_t)s, scan64, tot);
    const int64_t need = a.usage + carry + (int64_t)before + (s < 0 ? 0 : s) - a.capacity;
    uint32_t k = 0;
    if (need > 0) {
      uint32_t lo = 0, hi = nr;  // first index whose inclusive sum reaches need
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if ((int64_t)psum[mid] >= need) hi = mid; else lo = mid + 1;
      }
      k = lo < nr ? lo + 1 : nr;
    }
    if (j < a.n_demands) a.upto[j] = k;
    if (j == a.n_demands - 1) *last = k;
    carry += (int64_t)tot;  // (every thread holds the chunk's total)
    block_sync();
  }
  if (__ballot(bad) && lane_id() == 0) atomicOr(a.flags, kFlagRange);
  const uint32_t k_last = a.n_demands > 0 ? *last : 0;
  for (uint32_t e = t; e < k_last; e += BT) a.victims[e] = (int32_t)eorder[e];
}

struct EvictShared {
  uint64_t key[kEvictCap];
  uint32_t id[kEvictCap];
  uint32_t src[kEvictCap];    // index into the caller's cached / kv arrays
  uint64_t scan64[BT / kWave + 1];
  SortScratch sort;
  uint32_t bad;
};

__global__ __launch_bounds__(BT) void b_evict(EvictArgs a) {
  __shared__ EvictShared sh;
  const uint32_t t = threadIdx.x;
  const uint32_t nr = (uint32_t)a.n_cached;
  const uint32_t N = sort_size<true>(nr);
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
  sort_pairs<true>(sh.key, sh.id, sh.src, nr, sh.sort);
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
  evict_demands(a, sh.key, sh.id, nr, sh.scan64, &sh.bad);
}

// ---- lists beyond one workgroup's LDS -----------------------------------------
// The lists are sorted in chunks of kWideChunk entries, one workgroup each
// (the LDS sort above), and the sorted runs are then merged pairwise, one
// launch per round: an entry's place in the merged run is its index in its
// own run plus the number of entries of the other run before it, found by
// binary search (entries of the first run go before equal entries of the
// second, so the merge keeps the order of equal keys).

__device__ __forceinline__ int64_t list_size(const WideList& l) { return l.n0 + l.n1; }
__device__ __forceinline__ int64_t list_chunks(const WideList& l) {
  return (list_size(l) + kWideChunk - 1) / kWideChunk;
}

template <bool PAY>
struct ChunkShared {
  uint64_t key[kWideChunk];
  uint32_t id[kWideChunk];
  uint32_t pay[PAY ? kWideChunk : 1];
  SortScratch sort;
};

// PAY (eviction): entries carry their index in the caller's arrays, and a
// negative KV size is a range error. Ids outside [0, n_ids) are reported and
// sort last; the outputs of a call with an error are not written.
template <bool PAY>
__global__ __launch_bounds__(BT) void w_chunk_sort(WideSort a) {
  __shared__ ChunkShared<PAY> sh;
  __shared__ uint32_t s_bad;
  int64_t c = blockIdx.x;
  const bool second = a.nlists > 1 && c >= list_chunks(a.list[0]);
  const WideList l = second ? a.list[1] : a.list[0];
  if (second) c -= list_chunks(a.list[0]);
  const int64_t c0 = c * kWideChunk;
  const uint32_t nc = (uint32_t)min((int64_t)kWideChunk, list_size(l) - c0);
  const uint32_t t = threadIdx.x;
  if (t == 0) s_bad = 0;
  block_sync();
  uint32_t bad = 0;
  for (uint32_t i = t; i < nc; i += BT) {
    const int64_t gi = c0 + i;
    const int32_t v = gi < l.n0 ? l.src0[gi] : l.src1[gi - l.n0];
    uint64_t k = ~0ull;
    uint32_t id = ~0u;
    if (v < 0 || v >= a.n_ids) {
      bad |= 1u;
    } else if (PAY && a.kv[gi] < 0) {
      bad |= 2u;  // negative KV size
    } else {
      id = (uint32_t)v;
      k = (uint64_t)a.priority[id] << 32 | (uint32_t)a.length[id];
    }
    sh.key[i] = k;
    sh.id[i] = id;
    if (PAY) sh.pay[i] = (uint32_t)gi;
  }
  if (bad) atomicOr(&s_bad, bad);
  block_sync();
  if (t == 0 && s_bad) atomicOr(a.flags, (s_bad & 1u) ? kFlagInval : kFlagRange);
  block_sort<kWideChunk / BT, PAY>(sh.key, sh.id, sh.pay, nc, sh.sort);
  for (uint32_t i = t; i < nc; i += BT) {
    const int64_t o = l.base + c0 + i;
    a.key[0][o] = sh.key[i];
    a.id[0][o] = sh.id[i];
    if (PAY) a.pay[0][o] = sh.pay[i];
  }
}

// One merge round: runs of `run` entries (sorted) in buffer `from` become
// runs of 2 * run in the other buffer.
template <bool PAY>
__global__ __launch_bounds__(BT) void w_merge(WideSort a, int64_t run, int from) {
  const uint64_t* kin = a.key[from];
  const uint32_t* iin = a.id[from];
  const int to = from ^ 1;
  for (int64_t g = (int64_t)blockIdx.x * BT + threadIdx.x; g < a.total;
       g += (int64_t)gridDim.x * BT) {
    const bool second = a.nlists > 1 && g >= a.list[1].base;
    const int64_t base = second ? a.list[1].base : a.list[0].base;
    const int64_t n = list_size(second ? a.list[1] : a.list[0]);
    const int64_t i = g - base;
    const int64_t ps = i / (2 * run) * (2 * run);   // the pair's first entry
    const int64_t am = min(ps + run, n);             // end of its first run
    const int64_t be = min(ps + 2 * run, n);         // end of its second run
    const uint64_t k = kin[g];
    const uint32_t id = iin[g];
    int64_t pos;
    if (i < am)
      pos = i + count_below(kin + base + am, iin + base + am, (uint32_t)(be - am), k, id);
    else
      pos = ps + (i - am) + count_not_above(kin + base + ps, iin + base + ps, (uint32_t)(am - ps),
                                            k, id);
    a.key[to][base + pos] = k;
    a.id[to][base + pos] = id;
    if (PAY) a.pay[to][base + pos] = a.pay[from][g];
  }
}

// Selection on the sorted candidates (list 0; C = their first nc) and ongoing
// requests (list 1): the stage filter, the kept members of C before each
// index (dec), and the counts.
__global__ __launch_bounds__(BT) void w_select_scan(SelArgs a, WideSort w, int buf,
                                                    uint32_t* dec) {
  __shared__ uint32_t scan32[BT / kWave + 1];
  const uint32_t t = threadIdx.x;
  if (load_agent(a.flags) != 0) {  // an id outside [0, n_ids)
    if (t == 0) a.counts[0] = a.counts[1] = 0;
    return;
  }
  const uint64_t* ck = w.key[buf];
  const uint32_t* ci = w.id[buf];
  const uint64_t* ok = ck + w.list[1].base;
  const uint32_t* oi = ci + w.list[1].base;
  const uint32_t nc = (uint32_t)min(a.b, list_size(w.list[0]));
  const uint32_t no = (uint32_t)list_size(w.list[1]);
  if (nc == 0 && no == 0) {
    if (t == 0) a.counts[0] = a.counts[1] = 0;
    return;
  }
  const bool top_in_c = nc > 0 && (no == 0 || less(ck[0], ci[0], ok[0], oi[0]));
  const bool keep_all = a.stage[top_in_c ? ci[0] : oi[0]] == 0;
  const uint32_t per = (nc + BT - 1) / BT;
  const uint32_t c0 = min(nc, t * per), c1 = min(nc, c0 + per);
  uint32_t mine = 0;
  for (uint32_t i = c0; i < c1; ++i) mine += (keep_all || a.stage[ci[i]] != 0) ? 1u : 0u;
  uint32_t ndec;
  uint32_t run = block_excl_scan_u32<BT>(mine, scan32, ndec);
  for (uint32_t i = c0; i < c1; ++i) {
    dec[i] = run;
    run += (keep_all || a.stage[ci[i]] != 0) ? 1u : 0u;
  }
  if (t == 0) {
    dec[nc] = ndec;
    const uint64_t b = (uint64_t)a.b, nm = (uint64_t)ndec + no;
    a.counts[0] = (int64_t)min(b, nm);
    a.counts[1] = (int64_t)((nc - ndec) + (nm > b ? nm - b : 0));
  }
}

__global__ __launch_bounds__(BT) void w_select_place(SelArgs a, WideSort w, int buf,
                                                     const uint32_t* dec) {
  if (load_agent(a.flags) != 0) return;
  const uint64_t* ck = w.key[buf];
  const uint32_t* ci = w.id[buf];
  const uint32_t nc = (uint32_t)min(a.b, list_size(w.list[0]));
  const uint32_t no = (uint32_t)list_size(w.list[1]);
  for (uint32_t g = blockIdx.x * BT + threadIdx.x; g < nc + no; g += gridDim.x * BT)
    select_place(a, ck, ci, nc, ck + w.list[1].base, ci + w.list[1].base, no, dec, g);
}

// Eviction on the sorted cached requests: KV prefix sums in eviction order
// (the sorted order read backwards) and the eviction order itself, then the
// victims of every incoming request.
__global__ __launch_bounds__(BT) void w_evict(EvictArgs a, WideSort w, int buf, uint64_t* psum,
                                              uint32_t* eorder) {
  __shared__ uint64_t scan64[BT / kWave + 1];
  __shared__ uint32_t last;
  if (load_agent(a.flags) != 0) return;  // a bad id or KV size
  const uint32_t t = threadIdx.x;
  const uint32_t nr = (uint32_t)a.n_cached;
  const uint32_t* id = w.id[buf];
  const uint32_t* src = w.pay[buf];
  const uint32_t per = (nr + BT - 1) / BT;
  const uint32_t e0 = min(nr, t * per), e1 = min(nr, e0 + per);
  uint64_t mine = 0;
  for (uint32_t e = e0; e < e1; ++e) mine += (uint64_t)a.kv[src[nr - 1 - e]];
  uint64_t total;
  uint64_t run = block_excl_scan_u64<BT>(mine, scan64, total);
  for (uint32_t e = e0; e < e1; ++e) {
    run += (uint64_t)a.kv[src[nr - 1 - e]];
    psum[e] = run;            // KV evicted by the first e + 1 victims
    eorder[e] = id[nr - 1 - e];
  }
  block_sync();  // (orders this workgroup's global writes before its reads)
  evict_demands(a, psum, eorder, nr, scan64, &last);
}

// Chunk sort and merge rounds; returns the buffer that holds the result.
template <bool PAY>
int wide_sort(const WideSort& w, hipStream_t st) {
  int64_t chunks = 0, longest = 0;
  for (int l = 0; l < w.nlists; ++l) {
    const int64_t n = w.list[l].n0 + w.list[l].n1;
    chunks += (n + kWideChunk - 1) / kWideChunk;
    longest = std::max(longest, n);
  }
  if (chunks == 0) return 0;
  hipLaunchKernelGGL(w_chunk_sort<PAY>, dim3((unsigned)chunks), dim3(BT), 0, st, w);
  const unsigned grid = (unsigned)std::min<int64_t>((w.total + BT - 1) / BT, 4096);
  int from = 0;
  for (int64_t run = kWideChunk; run < longest; run *= 2) {
    hipLaunchKernelGGL(w_merge<PAY>, dim3(grid), dim3(BT), 0, st, w, run, from);
    from ^= 1;
  }
  return from;
}

}  // namespace

hipError_t launch_select_wide(const SelArgs& a, WideSort w, uint32_t* dec, hipStream_t st) {
  const int buf = wide_sort<false>(w, st);
  hipLaunchKernelGGL(w_select_scan, dim3(1), dim3(BT), 0, st, a, w, buf, dec);
  const int64_t nc = std::min(a.b, w.list[0].n0 + w.list[0].n1);
  const int64_t m = nc + w.list[1].n0 + w.list[1].n1;
  if (m > 0) {
    const unsigned grid = (unsigned)std::min<int64_t>((m + BT - 1) / BT, 4096);
    hipLaunchKernelGGL(w_select_place, dim3(grid), dim3(BT), 0, st, a, w, buf, dec);
  }
  return hipGetLastError();
}

hipError_t launch_evict_wide(const EvictArgs& a, WideSort w, uint64_t* psum, uint32_t* eorder,
                             hipStream_t st) {
  const int buf = wide_sort<true>(w, st);
  hipLaunchKernelGGL(w_evict, dim3(1), dim3(BT), 0, st, a, w, buf, psum, eorder);
  return hipGetLastError();
}

hipError_t launch_select(const SelArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(b_select, dim3(1), dim3(BT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_evict_victims(const EvictArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(b_evict, dim3(1), dim3(BT), 0, st, a);
  return hipGetLastError();
}

}  // namespace semsched
