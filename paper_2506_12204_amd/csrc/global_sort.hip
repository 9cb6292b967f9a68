// Multi-pass schedule of one long queue (n > SEM_SEGMENT_CAP).
//
// The schedule is the drained min-heap of Algorithm 1 (MinHeap
// Construction): ids ascending by (priority, length, id). Here it is an LSD
// radix sort over only the live bits of (priority, length), followed by the
// waits of Eq. 1 (the exclusive prefix of service times) and exact per-class
// totals, all fused into the last pass.
//
//   g_reset    clear the small per-call state and the totals.
//   g_hist     read (priority, length) once: validate, find the ranges and
//              count the low `d0` bits of every length. That digit does not
//              depend on the ranges, so no separate min/max pass is needed.
//              The last workgroup to finish writes the Plan.
//   g_scatter  one stable scatter pass per digit, with decoupled look-back
//              on per-tile digit counts. The first pass packs every request
//              into one u64 element  (p - pmin | (len >> d0) - hmin | len & lo
//              | id)  and scatters it by the low length digit. Middle passes
//              (rare: only for very wide key ranges) scatter by 10-bit digits
//              of u2 = (p - pmin) * H + h. The final pass scatters by the top
//              digit of u2 with a second, length-weighted look-back, so each
//              request's position AND wait come out of the same pass.
//
// Every scatter workgroup is persistent: it takes tile ids from an atomic
// counter, so a tile only ever waits (in the look-back) on tiles that were
// handed out earlier to running workgroups.
#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int NT = kGlobalThreads;
constexpr int K = kGlobalRounds;
constexpr int NW = NT / kWave;
constexpr int T = kGlobalTile;
constexpr int kBinsPerThread = (kMaxBins + NT - 1) / NT;
static_assert(kBinsPerThread * NT >= kMaxBins, "every bin has a thread");

constexpr uint32_t kAgg = 1;  // look-back flag: tile aggregate only
constexpr uint32_t kInc = 2;  // look-back flag: inclusive prefix over tiles

template <typename ST>
struct Status {
  static constexpr int SH = (int)sizeof(ST) * 8 - 2;
  static constexpr ST VMASK = (ST(1) << SH) - 1;
  static __device__ __forceinline__ ST make(uint32_t flag, uint64_t v) {
    return (ST(flag) << SH) | ST(v);
  }
};
using WStatus = Status<uint64_t>;

// ------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void g_reset(GArgs a) {
  const int t = threadIdx.x;
  if (t == 0) {
    a.flags[0] = 0;
    a.done[0] = 0;
    a.minmax[0] = 0xffu;        // pmin
    a.minmax[1] = 0;            // pmax
    a.minmax[2] = 0xffffffffu;  // lmin
    a.minmax[3] = 0;            // lmax
    a.plan->ok = 0;
  }
  if (t < kMaxScatter) a.tile_ctr[t] = 0;
  for (int i = t; i < kMaxScatter * kMaxBins; i += 1024) {
    a.hist_cnt[i] = 0;
    a.hist_w[i] = 0;
  }
  for (int i = t; i < 2 * (1 + a.num_classes); i += 1024) a.totals[i] = 0;
}

// ------------------------------------------------------------------------
constexpr int kHistThreads = 256;

__device__ __forceinline__ void hist_one(uint32_t p, int32_t l, int ncls, uint32_t mask,
                                         uint32_t* s_hist, uint32_t& lmin, uint32_t& lmax,
                                         uint32_t& pmin, uint32_t& pmax, uint32_t& bad) {
  if (l < 0 || (int)p >= ncls) {
    bad = 1;
    return;
  }
  lmin = min(lmin, (uint32_t)l);
  lmax = max(lmax, (uint32_t)l);
  pmin = min(pmin, p);
  pmax = max(pmax, p);
  atomicAdd(&s_hist[(uint32_t)l & mask], 1u);
}

__global__ __launch_bounds__(kHistThreads) void g_hist(GArgs a, int vec_ok) {
  constexpr int HW = kHistThreads / kWave;
  __shared__ uint32_t s_hist[kMaxBins];
  __shared__ uint32_t s_red[4][HW];
  __shared__ uint32_t s_last;
  const int t = threadIdx.x;
  const int nb = 1 << a.d0;
  const uint32_t mask = (uint32_t)nb - 1;
  for (int b = t; b < nb; b += kHistThreads) s_hist[b] = 0;
  block_sync();

  uint32_t lmin = 0xffffffffu, lmax = 0, pmin = 0xffu, pmax = 0, bad = 0;
  const int64_t stride = (int64_t)gridDim.x * kHistThreads;
  int64_t done_upto = 0;
  if (vec_ok) {
    const int64_t n4 = a.n / 4;
    const uint32_t* p4 = reinterpret_cast<const uint32_t*>(a.priority);
    const int4* l4 = reinterpret_cast<const int4*>(a.length);
    for (int64_t g = (int64_t)blockIdx.x * kHistThreads + t; g < n4; g += stride) {
      const uint32_t pv = p4[g];
      const int4 lv = l4[g];
      hist_one(pv & 0xff, lv.x, a.num_classes, mask, s_hist, lmin, lmax, pmin, pmax, bad);
      hist_one((pv >> 8) & 0xff, lv.y, a.num_classes, mask, s_hist, lmin, lmax, pmin, pmax, bad);
      hist_one((pv >> 16) & 0xff, lv.z, a.num_classes, mask, s_hist, lmin, lmax, pmin, pmax, bad);
      hist_one(pv >> 24, lv.w, a.num_classes, mask, s_hist, lmin, lmax, pmin, pmax, bad);
    }
    done_upto = n4 * 4;
  }
  for (int64_t i = done_upto + (int64_t)blockIdx.x * kHistThreads + t; i < a.n; i += stride)
    hist_one(a.priority[i], a.length[i], a.num_classes, mask, s_hist, lmin, lmax, pmin,
             pmax, bad);

  lmin = wave_min_u32(lmin);
  lmax = wave_max_u32(lmax);
  pmin = wave_min_u32(pmin);
  pmax = wave_max_u32(pmax);
  bad = wave_or_u32(bad);
  const int w = t / kWave;
  if (lane_id() == 0) {
    s_red[0][w] = lmin;
    s_red[1][w] = lmax;
    s_red[2][w] = pmin;
    s_red[3][w] = pmax | (bad << 31);
  }
  block_sync();
  if (t == 0) {
    for (int i = 1; i < HW; ++i) {
      lmin = min(lmin, s_red[0][i]);
      lmax = max(lmax, s_red[1][i]);
      pmin = min(pmin, s_red[2][i]);
      pmax = max(pmax, s_red[3][i] & 0xffu);
      bad |= s_red[3][i] >> 31;
    }
    lmin = min(lmin, s_red[0][0]);
    lmax = max(lmax, s_red[1][0]);
    pmin = min(pmin, s_red[2][0]);
    pmax = max(pmax, s_red[3][0] & 0xffu);
    bad |= s_red[3][0] >> 31;
    if (bad) atomicOr(a.flags, kFlagRange);
    atomicMin(&a.minmax[0], pmin);
    atomicMax(&a.minmax[1], pmax);
    atomicMin(&a.minmax[2], lmin);
    atomicMax(&a.minmax[3], lmax);
  }
  for (int b = t; b < nb; b += kHistThreads) {
    const uint32_t c = s_hist[b];
    if (c) atomicAdd(&a.hist_cnt[b], c);
  }

  // Clear the first scatter pass's look-back status (its size is fixed).
  {
    const size_t words = (size_t)a.tiles * nb * (a.wide_status ? 2 : 1);
    uint32_t* z = reinterpret_cast<uint32_t*>(a.cstat[0]);
    for (size_t i = (size_t)blockIdx.x * kHistThreads + t; i < words; i += stride) z[i] = 0;
  }

  // The last workgroup to finish turns the ranges into the Plan.
  __threadfence();
  block_sync();
  if (t == 0) s_last = (atomicAdd(a.done, 1u) == gridDim.x - 1) ? 1u : 0u;
  block_sync();
  if (!s_last || t != 0) return;
  __threadfence();
  const uint32_t fl = load_agent(a.flags);
  const uint32_t gpmin = load_agent(&a.minmax[0]);
  const uint32_t gpmax = load_agent(&a.minmax[1]);
  const uint32_t glmin = load_agent(&a.minmax[2]);
  const uint32_t glmax = load_agent(&a.minmax[3]);
  Plan* pl = a.plan;
  if (fl != 0) {
    pl->ok = 0;
    return;
  }
  const uint32_t d0 = (uint32_t)a.d0;
  const uint32_t P = gpmax - gpmin + 1;
  const uint32_t hmin = glmin >> d0;
  const uint32_t H = (glmax >> d0) - hmin + 1;
  const uint32_t wp = bit_width32(P - 1);
  const uint32_t wh = bit_width32(H - 1);
  const uint32_t W = bit_width32((uint32_t)(a.n - 1));
  pl->pmin = gpmin;
  pl->P = P;
  pl->hmin = hmin;
  pl->H = H;
  pl->wp = wp;
  pl->wh = wh;
  pl->W = W;
  pl->packed = (!a.force_wide && wp + wh + d0 + W <= 64) ? 1u : 0u;
  const uint64_t R = (uint64_t)P * H;  // <= 2^31 because d0 >= 8
  pl->shift[0] = 0;
  pl->nbits[0] = d0;
  pl->nbins[0] = 1u << d0;
  uint32_t mids = 0;
  if (R > (uint64_t)kMaxBins) {
    const uint32_t b2 = bit_width32((uint32_t)(R - 1));
    mids = (b2 - 10 + 9) / 10;
  }
  for (uint32_t s = 1; s <= mids; ++s) {
    pl->shift[s] = 10 * (s - 1);
    pl->nbits[s] = 10;
    pl->nbins[s] = kMaxBins;
  }
  const uint32_t sf = 10 * mids;
  const uint32_t fb = (uint32_t)((R - 1) >> sf) + 1;
  pl->shift[1 + mids] = sf;
  pl->nbins[1 + mids] = fb;
  pl->nbits[1 + mids] = bit_width32(fb - 1);
  pl->nscatter = 2 + mids;
  pl->ok = 1;
}

// ------------------------------------------------------------------------
// Scatter passes.

struct KeyCodec {
  uint32_t d0, wh, W, hmin, H, pmin;
  uint64_t m0, mh, idmask;
  __device__ __forceinline__ uint32_t lo(uint64_t key) const { return (uint32_t)(key & m0); }
  __device__ __forceinline__ uint32_t h(uint64_t key) const {
    return (uint32_t)((key >> d0) & mh);
  }
  __device__ __forceinline__ uint32_t pp(uint64_t key) const {
    return (uint32_t)(key >> (d0 + wh));
  }
  __device__ __forceinline__ uint32_t u2(uint64_t key) const { return pp(key) * H + h(key); }
  __device__ __forceinline__ uint32_t len(uint64_t key) const {
    return ((h(key) + hmin) << d0) | lo(key);
  }
  __device__ __forceinline__ uint64_t make(uint32_t p, uint32_t l) const {
    return ((uint64_t)(p - pmin) << (d0 + wh)) | ((uint64_t)((l >> d0) - hmin) << d0) |
           (l & (uint32_t)m0);
  }
};

struct FinShared {
  uint64_t gw[kMaxBins];
  uint64_t wfirst[kMaxBins];
  uint64_t wagg[kMaxBins];  // then the per-bin wait base
  uint64_t clo[256];
  uint64_t chi[256];
};
struct MidShared {
  uint32_t ncnt[kMaxBins];
  uint64_t nw[kMaxBins];
};

struct GShared {
  uint64_t stage[T];  // staged elements; the wave counters alias its front
  uint32_t excl[kMaxBins + 1];
  uint32_t base[kMaxBins];
  uint32_t gbase[kMaxBins];
  union {
    FinShared fin;
    MidShared mid;
  } u;
  uint64_t scan64[NW + 1];
  uint32_t scan32[NW + 1];
  uint32_t tile;
};
static_assert(NW * kMaxBins * 2 <= T * 8, "wave counters must fit in the stage");

template <bool FIRST, bool FINAL, typename ST>
__global__ __launch_bounds__(NT) void g_scatter(GArgs a, int s_arg) {
  static_assert(!(FIRST && FINAL), "at least two scatter passes");
  __shared__ GShared sh;
  uint16_t* cnt = reinterpret_cast<uint16_t*>(sh.stage);
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  const int S = (int)pl->nscatter;
  const int s = FINAL ? S - 1 : s_arg;
  if (!FIRST && !FINAL && s >= S - 1) return;  // this middle pass is not needed

  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
  const int nb = (int)pl->nbins[s];
  const int nbits = (int)pl->nbits[s];
  const uint32_t dshift = pl->shift[s];
  const uint32_t dmask = (1u << nbits) - 1;
  const bool next_final = !FINAL && (s + 1 == S - 1);
  const int nb_next = FINAL ? 0 : (int)pl->nbins[s + 1];
  const uint32_t nshift = FINAL ? 0 : pl->shift[s + 1];
  const uint32_t nmask = FINAL ? 0 : (1u << pl->nbits[s + 1]) - 1;

  KeyCodec kc;
  kc.d0 = (uint32_t)a.d0;
  kc.wh = pl->wh;
  kc.W = pl->W;
  kc.hmin = pl->hmin;
  kc.H = pl->H;
  kc.pmin = pl->pmin;
  kc.m0 = (1ull << kc.d0) - 1;
  kc.mh = (1ull << kc.wh) - 1;
  kc.idmask = (1ull << kc.W) - 1;
  const bool packed = pl->packed != 0;

  const uint64_t* keys_in = FIRST ? nullptr : a.keys[(s - 1) & 1];
  const uint32_t* ids_in = FIRST ? nullptr : a.ids[(s - 1) & 1];
  uint64_t* keys_out = FINAL ? nullptr : a.keys[s & 1];
  uint32_t* ids_out = FINAL ? nullptr : a.ids[s & 1];
  ST* cst = reinterpret_cast<ST*>(a.cstat[s & 1]);

  auto digit_of = [&](uint64_t key) -> uint32_t {
    return FIRST ? kc.lo(key) : ((kc.u2(key) >> dshift) & dmask);
  };

  // ---- per-kernel setup -------------------------------------------------
  if (!FINAL) {
    // clear the next pass's look-back status
    const size_t cwords = (size_t)a.tiles * nb_next * sizeof(ST) / 4;
    uint32_t* zc = reinterpret_cast<uint32_t*>(a.cstat[(s + 1) & 1]);
    const size_t stride = (size_t)gridDim.x * NT;
    for (size_t i = (size_t)blockIdx.x * NT + t; i < cwords; i += stride) zc[i] = 0;
    if (next_final) {
      const size_t n64 = (size_t)a.tiles * nb_next;
      for (size_t i = (size_t)blockIdx.x * NT + t; i < n64; i += stride) a.wstat[i] = 0;
    }
    for (int b = t; b < kMaxBins; b += NT) {
      sh.u.mid.ncnt[b] = 0;
      sh.u.mid.nw[b] = 0;
    }
  } else {
    for (int b = t; b < 256; b += NT) sh.u.fin.clo[b] = sh.u.fin.chi[b] = 0;
  }
  {
    // global digit bases: exclusive scan of the digit histogram, kBinsPerThread
    // consecutive bins per thread
    uint32_t c[kBinsPerThread];
    uint32_t csum = 0;
#pragma unroll
    for (int i = 0; i < kBinsPerThread; ++i) {
      const int b = t * kBinsPerThread + i;
      c[i] = b < nb ? a.hist_cnt[s * kMaxBins + b] : 0u;
      csum += c[i];
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan_u32<NT>(csum, sh.scan32, tot);
#pragma unroll
    for (int i = 0; i < kBinsPerThread; ++i) {
      const int b = t * kBinsPerThread + i;
      if (b < nb) sh.gbase[b] = ex;
      ex += c[i];
    }
    if (FINAL) {
      uint64_t wv[kBinsPerThread];
      uint64_t wsum = 0;
#pragma unroll
      for (int i = 0; i < kBinsPerThread; ++i) {
        const int b = t * kBinsPerThread + i;
        wv[i] = b < nb ? a.hist_w[s * kMaxBins + b] : 0ull;
        wsum += wv[i];
      }
      uint64_t wt;
      uint64_t wex = block_excl_scan_u64<NT>(wsum, sh.scan64, wt);
#pragma unroll
      for (int i = 0; i < kBinsPerThread; ++i) {
        const int b = t * kBinsPerThread + i;
        if (b < nb) sh.u.fin.gw[b] = wex;
        wex += wv[i];
      }
    }
  }

  // ---- tiles ------------------------------------------------------------
  for (;;) {
    block_sync();
    if (t == 0) sh.tile = atomicAdd(&a.tile_ctr[s], 1u);
    block_sync();
    const int tile = (int)sh.tile;
    if (tile >= a.tiles) break;
    const int64_t tb = (int64_t)tile * T;
    const int cv = (int)min((int64_t)T, a.n - tb);
    const int wb = w * kWave * K;

    uint64_t key[K];
    uint32_t id[K], dg[K], rk[K];
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int il = wb + r * kWave + lane;
      key[r] = 0;
      id[r] = 0;
      dg[r] = (uint32_t)nb - 1;  // invalid items sit last and sort last
      if (il < cv) {
        const int64_t i = tb + il;
        uint32_t len;
        if (FIRST) {
          const uint32_t p = a.priority[i];
          len = (uint32_t)a.length[i];
          key[r] = kc.make(p, len);
          id[r] = (uint32_t)i;
        } else if (packed) {
          const uint64_t e = keys_in[i];
          key[r] = e >> kc.W;
          id[r] = (uint32_t)(e & kc.idmask);
          len = kc.len(key[r]);
        } else {
          key[r] = keys_in[i];
          id[r] = ids_in[i];
          len = kc.len(key[r]);
        }
        dg[r] = digit_of(key[r]);
        if (!FINAL) {
          const uint32_t dn = (kc.u2(key[r]) >> nshift) & nmask;
          atomicAdd(&sh.u.mid.ncnt[dn], 1u);
          if (next_final) atomicAdd((unsigned long long*)&sh.u.mid.nw[dn], (unsigned long long)len);
        }
      }
    }

    // stable rank inside the tile
    for (int b = lane; b < nb; b += kWave) cnt[w * kMaxBins + b] = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) rk[r] = rank_round(dg[r], nbits, cnt + w * kMaxBins);
    block_sync();
    block_digit_offsets<NT>(cnt, kMaxBins, nb, sh.excl, sh.scan32);
#pragma unroll
    for (int r = 0; r < K; ++r) rk[r] += sh.excl[dg[r]] + cnt[w * kMaxBins + dg[r]];

    if (!FINAL) {
      // decoupled look-back on digit counts, bins spread over the threads
      for (int b = t; b < nb; b += NT) {
        const uint64_t agg = sh.excl[b + 1] - sh.excl[b];
        uint64_t ex = 0;
        if (tile == 0) {
          store_agent(&cst[b], Status<ST>::make(kInc, agg));
        } else {
          store_agent(&cst[(size_t)tile * nb + b], Status<ST>::make(kAgg, agg));
          for (int j = tile - 1; j >= 0;) {
            const ST v = load_agent(&cst[(size_t)j * nb + b]);
            const uint32_t f = (uint32_t)(v >> Status<ST>::SH);
            if (f == 0) {
              __builtin_amdgcn_s_sleep(1);
              continue;
            }
            ex += (uint64_t)(v & Status<ST>::VMASK);
            if (f == kInc) break;
            --j;
          }
          store_agent(&cst[(size_t)tile * nb + b], Status<ST>::make(kInc, ex + agg));
        }
        sh.base[b] = sh.gbase[b] + (uint32_t)ex - sh.excl[b];
      }
      block_sync();  // counters read, bases ready
      uint32_t jid[K];
      if (!packed) {
        uint32_t* sid = reinterpret_cast<uint32_t*>(sh.stage);
#pragma unroll
        for (int r = 0; r < K; ++r) sid[rk[r]] = id[r];
        block_sync();
#pragma unroll
        for (int r = 0; r < K; ++r) jid[r] = sid[wb + r * kWave + lane];
        block_sync();
      }
#pragma unroll
      for (int r = 0; r < K; ++r)
        sh.stage[rk[r]] = packed ? ((key[r] << kc.W) | id[r]) : key[r];
      block_sync();
#pragma unroll
      for (int r = 0; r < K; ++r) {
        const int j = wb + r * kWave + lane;
        if (j < cv) {
          const uint64_t e = sh.stage[j];
          const uint64_t kj = packed ? (e >> kc.W) : e;
          const uint32_t pos = sh.base[digit_of(kj)] + (uint32_t)j;
          if (pos < (uint64_t)a.n) {  // always true for consistent counts
            keys_out[pos] = e;
            if (!packed) ids_out[pos] = jid[r];
          }
        }
      }
      continue;
    }

    // ---- final pass: positions, waits and totals ------------------------
    block_sync();  // counters read before the stage is written
    uint32_t js[K];
    if (!packed) {
      uint32_t* sid = reinterpret_cast<uint32_t*>(sh.stage);
#pragma unroll
      for (int r = 0; r < K; ++r) sid[rk[r]] = id[r];
      block_sync();
#pragma unroll
      for (int r = 0; r < K; ++r) js[r] = sid[wb + r * kWave + lane];
      block_sync();
    }
#pragma unroll
    for (int r = 0; r < K; ++r)
      sh.stage[rk[r]] = packed ? ((key[r] << kc.W) | id[r]) : key[r];
    block_sync();
    uint64_t ks[K], ls[K];
    uint64_t wsum = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      ks[r] = 0;
      ls[r] = 0;
      dg[r] = (uint32_t)nb - 1;
      if (j < cv) {
        const uint64_t e = sh.stage[j];
        ks[r] = packed ? (e >> kc.W) : e;
        if (packed) js[r] = (uint32_t)(e & kc.idmask);
        ls[r] = kc.len(ks[r]);
        dg[r] = digit_of(ks[r]);
      }
      wsum += ls[r];
    }
    uint64_t wtot = wave_incl_scan_u64(wsum);
    wtot = __shfl(wtot, kWave - 1, kWave);
    uint64_t dummy;
    uint64_t run = block_excl_scan_u64<NT>(lane == 0 ? wtot : 0, sh.scan64, dummy);
    run = __shfl(run, 0, kWave);
    uint64_t ex_w[K];  // exclusive length prefix inside the tile's sorted order
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const uint64_t incl = wave_incl_scan_u64(ls[r]);
      ex_w[r] = run + incl - ls[r];
      run += __shfl(incl, kWave - 1, kWave);
      const int j = wb + r * kWave + lane;
      if (j < cv && (uint32_t)j == sh.excl[dg[r]]) sh.u.fin.wfirst[dg[r]] = ex_w[r];
    }
    block_sync();
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      if (j < cv) {
        const int last = min((int)sh.excl[dg[r] + 1], cv) - 1;
        if (j == last) sh.u.fin.wagg[dg[r]] = ex_w[r] + ls[r] - sh.u.fin.wfirst[dg[r]];
      }
    }
    block_sync();
    for (int b = t; b < nb; b += NT) {
      const uint32_t e0 = sh.excl[b], e1 = sh.excl[b + 1];
      const bool any = min((int)e0, cv) < min((int)e1, cv);
      const uint64_t cagg = e1 - e0;
      const uint64_t wagg = any ? sh.u.fin.wagg[b] : 0ull;
      uint64_t cex = 0, wex = 0;
      if (tile == 0) {
        store_agent(&a.wstat[b], WStatus::make(kInc, wagg));
        store_agent(&cst[b], Status<ST>::make(kInc, cagg));
      } else {
        const size_t me = (size_t)tile * nb + b;
        store_agent(&a.wstat[me], WStatus::make(kAgg, wagg));
        store_agent(&cst[me], Status<ST>::make(kAgg, cagg));
        for (int j = tile - 1; j >= 0;) {
          const size_t at = (size_t)j * nb + b;
          const ST cv_ = load_agent(&cst[at]);
          const uint64_t wv = load_agent(&a.wstat[at]);
          const uint32_t cf = (uint32_t)(cv_ >> Status<ST>::SH);
          const uint32_t wf = (uint32_t)(wv >> WStatus::SH);
          if (cf == 0 || cf != wf) {
            __builtin_amdgcn_s_sleep(1);
            continue;
          }
          cex += (uint64_t)(cv_ & Status<ST>::VMASK);
          wex += wv & WStatus::VMASK;
          if (cf == kInc) break;
          --j;
        }
        store_agent(&a.wstat[me], WStatus::make(kInc, wex + wagg));
        store_agent(&cst[me], Status<ST>::make(kInc, cex + cagg));
      }
      sh.base[b] = sh.gbase[b] + (uint32_t)cex - e0;
      sh.u.fin.wagg[b] = sh.u.fin.gw[b] + wex - (any ? sh.u.fin.wfirst[b] : 0ull);
    }
    block_sync();
    int cur = -1;
    U128 acc = {0, 0};
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      if (j < cv) {
        const uint32_t pos = sh.base[dg[r]] + (uint32_t)j;
        const uint64_t wt = sh.u.fin.wagg[dg[r]] + ex_w[r];
        if (pos < (uint64_t)a.n) {  // always true for consistent counts
          a.wait[pos] = (int64_t)wt;
          a.order[pos] = (int32_t)js[r];
        }
        const int cls = (int)(kc.pp(ks[r]) + kc.pmin);
        if (cls != cur) {
          if (cur >= 0 && (acc.lo | acc.hi))
            atomic_add128(sh.u.fin.clo + cur, sh.u.fin.chi + cur, acc);
          cur = cls;
          acc.lo = acc.hi = 0;
        }
        add128(acc, wt);
      }
    }
    if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.u.fin.clo + cur, sh.u.fin.chi + cur, acc);
  }

  // ---- per-kernel teardown ------------------------------------------------
  block_sync();
  if (!FINAL) {
    for (int b = t; b < nb_next; b += NT) {
      const uint32_t c = sh.u.mid.ncnt[b];
      if (c) atomicAdd(&a.hist_cnt[(s + 1) * kMaxBins + b], c);
      if (next_final) {
        const uint64_t v = sh.u.mid.nw[b];
        if (v) atomicAdd((unsigned long long*)&a.hist_w[(s + 1) * kMaxBins + b],
                         (unsigned long long)v);
      }
    }
  } else {
    for (int c = t; c < a.num_classes; c += NT) {
      U128 v = {sh.u.fin.clo[c], sh.u.fin.chi[c]};
      if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + c), a.totals + 2 * (1 + c) + 1, v);
    }
    if (t == 0) {
      U128 g = {0, 0};
      for (int c = 0; c < 256; ++c) {
        U128 v = {sh.u.fin.clo[c], sh.u.fin.chi[c]};
        add128(g, v);
      }
      if (g.lo | g.hi) atomic_add128(a.totals, a.totals + 1, g);
    }
  }
}

__global__ void g_fill_zero(uint32_t* p, size_t count) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = 0;
}

int g_resident_grid() {
  static int cached = 0;
  if (cached) return cached;
  int dev = 0, cus = 256, occ = 1;
  if (hipGetDevice(&dev) == hipSuccess) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) cus = prop.multiProcessorCount;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &occ, reinterpret_cast<const void*>(g_scatter<false, true, uint32_t>), NT, 0) !=
          hipSuccess ||
      occ < 1)
    occ = 1;
  cached = cus * occ;
  return cached;
}

void mark(const StageEvents* ev, int stage, bool after, hipStream_t st) {
  if (!ev) return;
  hipEvent_t e = after ? ev->after[stage] : ev->before[stage];
  if (e) (void)hipEventRecord(e, st);
}

template <typename ST>
hipError_t launch_passes(const GArgs& a, hipStream_t st, const StageEvents* ev) {
  const int resident = g_resident_grid();
  const int grid = a.tiles < resident ? a.tiles : resident;
  mark(ev, 1, false, st);
  hipLaunchKernelGGL((g_scatter<true, false, ST>), dim3(grid), dim3(NT), 0, st, a, 0);
  mark(ev, 1, true, st);
  for (int s = 1; s < kMaxScatter - 1; ++s)
    hipLaunchKernelGGL((g_scatter<false, false, ST>), dim3(grid), dim3(NT), 0, st, a, s);
  mark(ev, 2, false, st);
  hipLaunchKernelGGL((g_scatter<false, true, ST>), dim3(grid), dim3(NT), 0, st, a, 0);
  mark(ev, 2, true, st);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_global_schedule(const GArgs& a, hipStream_t st, const StageEvents* ev) {
  hipLaunchKernelGGL(g_reset, dim3(1), dim3(1024), 0, st, a);
  const int vec_ok = ((uintptr_t)a.priority % 4 == 0) && ((uintptr_t)a.length % 16 == 0);
  int hgrid = (int)((a.n + 4 * kHistThreads * 8 - 1) / (4 * kHistThreads * 8));
  if (hgrid > 2048) hgrid = 2048;
  if (hgrid < 1) hgrid = 1;
  mark(ev, 0, false, st);
  hipLaunchKernelGGL(g_hist, dim3(hgrid), dim3(kHistThreads), 0, st, a, vec_ok);
  mark(ev, 0, true, st);
  if (a.wide_status) return launch_passes<uint64_t>(a, st, ev);
  return launch_passes<uint32_t>(a, st, ev);
}

hipError_t launch_fill_zero(uint32_t* p, size_t count, hipStream_t st) {
  if (count == 0) return hipSuccess;
  size_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(g_fill_zero, dim3((unsigned)blocks), dim3(256), 0, st, p, count);
  return hipGetLastError();
}

}  // namespace semsched
