// Multi-pass schedule of one long queue (n > SEM_SEGMENT_CAP).
//
// The schedule is the drained min-heap of Algorithm 1 (MinHeap
// Construction): ids ascending by (priority, length, id). Here it is an LSD
// radix sort over only the live bits of (priority, length), followed by the
// waits of Eq. 1 (the exclusive prefix of service times) and exact per-class
// totals, all fused into the last pass.
//
// Every pass splits the queue into the same blocks of consecutive tiles, one
// block per workgroup. A pass first counts the digits of every block, a
// column scan turns the counts into per-block offsets, and the scatter then
// walks its block tile by tile with running per-digit offsets. No workgroup
// ever waits for another inside a kernel, and consecutive tiles of a digit
// land next to each other in memory, written by the same workgroup.
//
//   g_reset   clear the small per-call state and the totals.
//   g_hist0   read (priority, length) once: validate, find the ranges and
//             count the low `d0` bits of every length per block. That digit
//             does not depend on the ranges, so no separate min/max pass is
//             needed.
//   g_scan    per-block digit offsets of one pass (column scans); for the
//             first pass one more workgroup reduces the block ranges into
//             the Plan.
//   g_first   first scatter pass: packs every request into one u64 element
//               (p - pmin | (len >> d0) - hmin | len & (2^d0 - 1) | id)
//             and scatters it by the low length digit.
//   g_mid     middle passes, only for very wide key ranges: count, scan and
//             scatter by 10-bit digits of u2 = (p - pmin) * H + h, in one
//             launch of co-resident workgroups with grid barriers between the
//             phases; it returns at once when two passes suffice.
//   g_histF   counts and length sums of the final digit per block.
//   g_final   final scatter by the top digit of u2 with running count and
//             length offsets: each request's position and wait come out of
//             the same pass, plus the per-class totals.
#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int NT = kGlobalThreads;
constexpr int K = kGlobalRounds;
constexpr int NW = NT / kWave;
constexpr int T = kGlobalTile;
constexpr int BPT = kMaxBins / NT;  // bins per thread, blocked: t*BPT .. t*BPT+BPT-1
static_assert(BPT * NT == kMaxBins, "every bin has a thread");
static_assert(NW * kMaxBins * 2 <= T * 8, "wave counters must fit in the stage");

// ------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void g_reset(GArgs a) {
  const int t = threadIdx.x;
  if (t == 0) {
    a.flags[0] = 0;
    a.barrier[0] = 0;
    a.plan->ok = 0;
  }
  for (int i = t; i < kMaxScatter * kMaxBins; i += 1024) a.hist_cnt[i] = 0;
  for (int i = t; i < kMaxBins; i += 1024) a.hist_w[i] = 0;
  for (int i = t; i < 2 * (1 + a.num_classes); i += 1024) a.totals[i] = 0;
}

// ------------------------------------------------------------------------
// Pass 0: ranges, validation and the first digit's per-block histogram.

constexpr int HT = 512;  // threads of the histogram passes
constexpr int SCT = 256;  // threads of the column scans
constexpr int SCT_WAVES = SCT / kWave;
constexpr int HU = 8;    // loads in flight per thread

struct Ranges {
  uint32_t lmin = 0xffffffffu, lmax = 0, pmin = 0xffu, pmax = 0, bad = 0;
  __device__ __forceinline__ void add(uint32_t p, int32_t l, int ncls, uint32_t mask,
                                      uint32_t* s_hist) {
    const bool ok = (l >= 0) & ((int)p < ncls);
    bad |= ok ? 0u : 1u;
    lmin = min(lmin, ok ? (uint32_t)l : 0xffffffffu);
    lmax = max(lmax, ok ? (uint32_t)l : 0u);
    pmin = min(pmin, ok ? p : 0xffu);
    pmax = max(pmax, ok ? p : 0u);
    atomicAdd(&s_hist[(uint32_t)l & mask], ok ? 1u : 0u);
  }
};

// Reduce the block ranges and turn them into the Plan (one workgroup).
__device__ void write_plan(const GArgs& a, int G) {
  __shared__ uint32_t s_red[4][SCT_WAVES];
  uint32_t pl_ = 0xffu, ph = 0, ll = 0xffffffffu, lh = 0;
  for (int g = threadIdx.x; g < G; g += SCT) {
    const uint32_t* r = a.block_ranges + 4 * (size_t)g;
    pl_ = min(pl_, r[0]);
    ph = max(ph, r[1]);
    ll = min(ll, r[2]);
    lh = max(lh, r[3]);
  }
  pl_ = wave_min_u32(pl_);
  ph = wave_max_u32(ph);
  ll = wave_min_u32(ll);
  lh = wave_max_u32(lh);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    s_red[0][w] = pl_;
    s_red[1][w] = ph;
    s_red[2][w] = ll;
    s_red[3][w] = lh;
  }
  block_sync();
  if (threadIdx.x != 0) return;
  uint32_t gpmin = 0xffu, gpmax = 0, glmin = 0xffffffffu, glmax = 0;
  for (int i = 0; i < SCT_WAVES; ++i) {
    gpmin = min(gpmin, s_red[0][i]);
    gpmax = max(gpmax, s_red[1][i]);
    glmin = min(glmin, s_red[2][i]);
    glmax = max(glmax, s_red[3][i]);
  }
  Plan* pl = a.plan;
  if (load_agent(a.flags) != 0) {
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

__global__ __launch_bounds__(HT) void g_hist0(GArgs a, int vec_ok) {
  constexpr int HW = HT / kWave;
  __shared__ uint32_t s_hist[kMaxBins];
  __shared__ uint32_t s_red[4][HW];
  const int t = threadIdx.x;
  const int g = blockIdx.x;
  const int nb = 1 << a.d0;
  const uint32_t mask = (uint32_t)nb - 1;
  for (int b = t; b < nb; b += HT) s_hist[b] = 0;
  block_sync();

  const int64_t lo = (int64_t)g * a.main.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)a.main.tpb * T);
  Ranges rg;
  int64_t scalar_from = lo;
  if (vec_ok && hi > lo) {
    const int64_t q0 = lo >> 2, q1 = hi >> 2;  // lo is a multiple of 4
    const uint32_t* p4 = reinterpret_cast<const uint32_t*>(a.priority);
    const int4* l4 = reinterpret_cast<const int4*>(a.length);
    for (int64_t q = q0 + t; q < q1; q += (int64_t)HT * HU) {
      uint32_t pv[HU];
      int4 lv[HU];
#pragma unroll
      for (int u = 0; u < HU; ++u) {
        const int64_t qq = min(q + (int64_t)u * HT, q1 - 1);  // in bounds; duplicates ignored
        pv[u] = p4[qq];
        lv[u] = l4[qq];
      }
#pragma unroll
      for (int u = 0; u < HU; ++u) {
        if (q + (int64_t)u * HT < q1) {
          rg.add(pv[u] & 0xff, lv[u].x, a.num_classes, mask, s_hist);
          rg.add((pv[u] >> 8) & 0xff, lv[u].y, a.num_classes, mask, s_hist);
          rg.add((pv[u] >> 16) & 0xff, lv[u].z, a.num_classes, mask, s_hist);
          rg.add(pv[u] >> 24, lv[u].w, a.num_classes, mask, s_hist);
        }
      }
    }
    scalar_from = q1 * 4;
  }
  for (int64_t i = scalar_from + t; i < hi; i += HT)
    rg.add(a.priority[i], a.length[i], a.num_classes, mask, s_hist);

  const uint32_t lmin = wave_min_u32(rg.lmin), lmax = wave_max_u32(rg.lmax);
  const uint32_t pmin = wave_min_u32(rg.pmin), pmax = wave_max_u32(rg.pmax);
  const uint32_t bad = wave_or_u32(rg.bad);
  const int w = t / kWave;
  if (lane_id() == 0) {
    s_red[0][w] = lmin;
    s_red[1][w] = lmax;
    s_red[2][w] = pmin;
    s_red[3][w] = pmax | (bad << 31);
  }
  block_sync();
  if (t == 0) {
    uint32_t bl = 0xffffffffu, bh = 0, pl = 0xffu, ph = 0, bb = 0;
    for (int i = 0; i < HW; ++i) {
      bl = min(bl, s_red[0][i]);
      bh = max(bh, s_red[1][i]);
      pl = min(pl, s_red[2][i]);
      ph = max(ph, s_red[3][i] & 0xffu);
      bb |= s_red[3][i] >> 31;
    }
    if (bb) atomicOr(a.flags, kFlagRange);
    uint32_t* r = a.block_ranges + 4 * (size_t)g;
    r[0] = pl;  // an empty block leaves the neutral values
    r[1] = ph;
    r[2] = bl;
    r[3] = bh;
  }
  for (int b = t; b < nb; b += HT) a.block_hist[(size_t)g * kMaxBins + b] = s_hist[b];
}

// ------------------------------------------------------------------------
// Column scans: block_hist[g][b] becomes the count of digit b in blocks
// before g (block_histw likewise for length sums); the totals go to
// hist_cnt[s][b] (and hist_w[b]).

template <int THREADS>
__device__ void column_scan(const GArgs& a, int s, int b, bool weights, int G,
                            uint32_t* scan32, uint64_t* scan64) {
  constexpr int SCPER = kMaxBlocks / THREADS;
  const int per = (G + THREADS - 1) / THREADS;
  const int g0 = (int)threadIdx.x * per;
  uint32_t v[SCPER];
  uint32_t local = 0;
#pragma unroll
  for (int i = 0; i < SCPER; ++i) {
    v[i] = 0;
    if (i < per && g0 + i < G) v[i] = a.block_hist[(size_t)(g0 + i) * kMaxBins + b];
    local += v[i];
  }
  uint32_t total;
  uint32_t run = block_excl_scan_u32<THREADS>(local, scan32, total);
#pragma unroll
  for (int i = 0; i < SCPER; ++i) {
    if (i < per && g0 + i < G) a.block_hist[(size_t)(g0 + i) * kMaxBins + b] = run;
    run += v[i];
  }
  if (threadIdx.x == 0) a.hist_cnt[s * kMaxBins + b] = total;
  if (!weights) return;
  uint64_t wv[SCPER];
  uint64_t wl = 0;
#pragma unroll
  for (int i = 0; i < SCPER; ++i) {
    wv[i] = 0;
    if (i < per && g0 + i < G) wv[i] = a.block_histw[(size_t)(g0 + i) * kMaxBins + b];
    wl += wv[i];
  }
  uint64_t wtot;
  uint64_t wrun = block_excl_scan_u64<THREADS>(wl, scan64, wtot);
#pragma unroll
  for (int i = 0; i < SCPER; ++i) {
    if (i < per && g0 + i < G) a.block_histw[(size_t)(g0 + i) * kMaxBins + b] = wrun;
    wrun += wv[i];
  }
  if (threadIdx.x == 0) a.hist_w[b] = wtot;
}

// final != 0: scan the final pass (its index and bin count come from the Plan).
// Pass 0 (final == 0): workgroups 0 .. 2^d0-1 scan the first digit's bins
// and workgroup 2^d0 writes the Plan. Final pass: one workgroup per bin.
__global__ __launch_bounds__(SCT) void g_scan(GArgs a, int final) {
  __shared__ uint32_t scan32[SCT / kWave + 1];
  __shared__ uint64_t scan64[SCT / kWave + 1];
  const int b = blockIdx.x;
  if (!final) {
    if (b == (1 << a.d0)) {
      write_plan(a, a.main.blocks);
      return;
    }
    column_scan<SCT>(a, 0, b, false, a.main.blocks, scan32, scan64);
    return;
  }
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  const int s = (int)pl->nscatter - 1;
  if (b >= (int)pl->nbins[s]) return;
  column_scan<SCT>(a, s, b, true, a.main.blocks, scan32, scan64);
}

// ------------------------------------------------------------------------
// Scatter passes.

struct KeyCodec {
  uint32_t d0, wh, W, hmin, H, pmin;
  uint64_t m0, mh, idmask;
  __device__ __forceinline__ void init(const GArgs& a, const Plan* pl) {
    d0 = (uint32_t)a.d0;
    wh = pl->wh;
    W = pl->W;
    hmin = pl->hmin;
    H = pl->H;
    pmin = pl->pmin;
    m0 = (1ull << d0) - 1;
    mh = (1ull << wh) - 1;
    idmask = (1ull << W) - 1;
  }
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

// Stable rank of the tile's K rounds by digit: on return rk[r] is the position
// of item (wave, round r, lane) in the tile's digit-sorted order and excl[b]
// the number of the tile's items with digit < b.
__device__ __forceinline__ void rank_tile(const uint32_t (&dg)[K], uint32_t (&rk)[K],
                                          int nb, int nbits, uint16_t* cnt, uint32_t* excl,
                                          uint32_t* scan32) {
  const int w = threadIdx.x / kWave;
  for (int b = lane_id(); b < nb; b += kWave) cnt[w * kMaxBins + b] = 0;
#pragma unroll
  for (int r = 0; r < K; ++r) rk[r] = rank_round(dg[r], nbits, cnt + w * kMaxBins);
  block_sync();
  block_digit_offsets<NT>(cnt, kMaxBins, nb, excl, scan32);
#pragma unroll
  for (int r = 0; r < K; ++r) rk[r] += excl[dg[r]] + cnt[w * kMaxBins + dg[r]];
}

// Global digit bases of pass s (exclusive scan of its digit totals) plus this
// block's offset, for this thread's BPT bins.
__device__ __forceinline__ void start_offsets(const GArgs& a, int s, int nb, int g,
                                              uint32_t (&carry)[BPT], uint32_t* scan32) {
  uint32_t c[BPT];
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int b = threadIdx.x * BPT + i;
    c[i] = b < nb ? a.hist_cnt[s * kMaxBins + b] : 0u;
    sum += c[i];
  }
  uint32_t tot;
  uint32_t ex = block_excl_scan_u32<NT>(sum, scan32, tot);
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int b = threadIdx.x * BPT + i;
    carry[i] = ex + (b < nb ? a.block_hist[(size_t)g * kMaxBins + b] : 0u);
    ex += c[i];
  }
}

// Stage the tile's elements at their ranks and scatter them to `pos` = base
// of their digit + staged index. Wide layout: ids travel in their own array.
template <typename DigitFn>
__device__ __forceinline__ void stage_and_scatter(uint64_t* stage, const uint32_t* base,
                                                  const uint64_t (&key)[K],
                                                  const uint32_t (&id)[K],
                                                  const uint32_t (&rk)[K], int cv, bool packed,
                                                  uint32_t W, int64_t n, uint64_t* keys_out,
                                                  uint32_t* ids_out, DigitFn digit_of) {
  const int wb = (threadIdx.x / kWave) * kWave * K;
  const int lane = lane_id();
  uint32_t jid[K];
  if (!packed) {
    uint32_t* sid = reinterpret_cast<uint32_t*>(stage);
#pragma unroll
    for (int r = 0; r < K; ++r) sid[rk[r]] = id[r];
    block_sync();
#pragma unroll
    for (int r = 0; r < K; ++r) jid[r] = sid[wb + r * kWave + lane];
    block_sync();
  }
#pragma unroll
  for (int r = 0; r < K; ++r) stage[rk[r]] = packed ? ((key[r] << W) | id[r]) : key[r];
  block_sync();
#pragma unroll
  for (int r = 0; r < K; ++r) {
    const int j = wb + r * kWave + lane;
    if (j < cv) {
      const uint64_t e = stage[j];
      const uint32_t pos = base[digit_of(packed ? (e >> W) : e)] + (uint32_t)j;
      if (pos < (uint64_t)n) {  // always true for consistent counts
        keys_out[pos] = e;
        if (!packed) ids_out[pos] = jid[r];
      }
    }
  }
}

struct ScatterShared {
  uint64_t stage[T];  // staged elements; the wave counters alias its front
  uint32_t excl[kMaxBins + 1];
  uint32_t base[kMaxBins];
  uint32_t scan32[NW + 1];
};

// One block of a first (s == 0) or middle scatter pass.
template <bool FIRST>
__device__ void scatter_block(const GArgs& a, int s, int g, Split sp, ScatterShared& sh) {
  uint16_t* cnt = reinterpret_cast<uint16_t*>(sh.stage);
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
  const int nb = (int)pl->nbins[s];
  const int nbits = (int)pl->nbits[s];
  const uint32_t dshift = pl->shift[s];
  const uint32_t dmask = (1u << nbits) - 1;
  KeyCodec kc;
  kc.init(a, pl);
  const bool packed = pl->packed != 0;
  const uint64_t* keys_in = FIRST ? nullptr : a.keys[(s - 1) & 1];
  const uint32_t* ids_in = FIRST ? nullptr : a.ids[(s - 1) & 1];
  auto digit_of = [&](uint64_t k) -> uint32_t {
    return FIRST ? kc.lo(k) : ((kc.u2(k) >> dshift) & dmask);
  };

  uint32_t carry[BPT];  // running output offset of each of this thread's digits
  start_offsets(a, s, nb, g, carry, sh.scan32);
  const int tile0 = g * sp.tpb;
  const int tile1 = min(a.tiles, tile0 + sp.tpb);
  for (int tile = tile0; tile < tile1; ++tile) {
    block_sync();
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
        if (FIRST) {
          key[r] = kc.make(a.priority[i], (uint32_t)a.length[i]);
          id[r] = (uint32_t)i;
        } else if (packed) {
          const uint64_t e = keys_in[i];
          key[r] = e >> kc.W;
          id[r] = (uint32_t)(e & kc.idmask);
        } else {
          key[r] = keys_in[i];
          id[r] = ids_in[i];
        }
        dg[r] = digit_of(key[r]);
      }
    }
    rank_tile(dg, rk, nb, nbits, cnt, sh.excl, sh.scan32);
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int b = t * BPT + i;
      if (b < nb) {
        sh.base[b] = carry[i] - sh.excl[b];
        carry[i] += sh.excl[b + 1] - sh.excl[b];
      }
    }
    block_sync();  // counters read and bases written before the stage is reused
    stage_and_scatter(sh.stage, sh.base, key, id, rk, cv, packed, kc.W, a.n, a.keys[s & 1],
                      a.ids[s & 1], digit_of);
  }
}

// 4 waves per SIMD: two 8-wave workgroups per CU, so one can compute while
// the other waits on memory.
constexpr int kScatterWavesPerSimd = 4;

template <typename unused = void>
__global__ __launch_bounds__(NT, kScatterWavesPerSimd) void g_first(GArgs a) {
  __shared__ ScatterShared sh;
  if (!a.plan->ok) return;
  scatter_block<true>(a, 0, blockIdx.x, a.main, sh);
}

// Per-block digit counts (and length sums) of pass s over its input elements.
struct CountShared {
  uint32_t cnt[kMaxBins];
  uint64_t w[kMaxBins];
};

__device__ void count_block(const GArgs& a, int s, int g, Split sp, bool weights,
                            CountShared& sh, int threads) {
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int nb = (int)pl->nbins[s];
  const uint32_t dshift = pl->shift[s];
  const uint32_t dmask = (1u << pl->nbits[s]) - 1;
  KeyCodec kc;
  kc.init(a, pl);
  const bool packed = pl->packed != 0;
  const uint64_t* keys_in = a.keys[(s - 1) & 1];
  for (int b = t; b < nb; b += threads) {
    sh.cnt[b] = 0;
    sh.w[b] = 0;
  }
  block_sync();
  const int64_t lo = (int64_t)g * sp.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)sp.tpb * T);
  // lo is even (a multiple of the tile), so pairs of elements stay aligned
  const int64_t q0 = lo >> 1, q1 = hi >> 1;
  const ulonglong2* k2 = reinterpret_cast<const ulonglong2*>(keys_in);
  auto add = [&](uint64_t e) {
    const uint64_t key = packed ? (e >> kc.W) : e;
    const uint32_t d = (kc.u2(key) >> dshift) & dmask;
    atomicAdd(&sh.cnt[d], 1u);
    if (weights) atomicAdd((unsigned long long*)&sh.w[d], (unsigned long long)kc.len(key));
  };
  for (int64_t q = q0 + t; q < q1; q += (int64_t)threads * HU) {
    ulonglong2 v[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) v[u] = k2[min(q + (int64_t)u * threads, q1 - 1)];
#pragma unroll
    for (int u = 0; u < HU; ++u) {
      if (q + (int64_t)u * threads < q1) {
        add(v[u].x);
        add(v[u].y);
      }
    }
  }
  if ((hi & 1) && t == 0 && hi > lo) add(keys_in[hi - 1]);
  block_sync();
  for (int b = t; b < nb; b += threads) {
    a.block_hist[(size_t)g * kMaxBins + b] = sh.cnt[b];
    if (weights) a.block_histw[(size_t)g * kMaxBins + b] = sh.w[b];
  }
}

__global__ __launch_bounds__(HT) void g_histF(GArgs a) {
  __shared__ CountShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  count_block(a, (int)pl->nscatter - 1, blockIdx.x, a.main, true, sh, HT);
}

// ---- middle passes: one launch of co-resident workgroups, grid barriers ----
union MidShared {
  ScatterShared scatter;
  CountShared count;
  struct {
    uint32_t scan32[NT / kWave + 1];
    uint64_t scan64[NT / kWave + 1];
  } scan;
};

// Grid barrier for a launch whose workgroups are all resident (the grid is
// sized to the occupancy limit). Arrival number k waits for k * gridDim.x
// arrivals. The wait is bounded: if the workgroups were ever not co-resident
// it gives up, records kFlagDevice and the kernel returns instead of hanging.
__device__ bool grid_barrier(const GArgs& a, uint32_t generation) {
  __shared__ uint32_t s_ok;
  __threadfence();  // every thread releases its global writes at agent scope
  block_sync();
  if (threadIdx.x == 0) {
    atomicAdd(a.barrier, 1u);
    const uint32_t target = generation * gridDim.x;
    uint32_t ok = 1;
    for (uint32_t spin = 0; load_agent(a.barrier) < target; ++spin) {
      if (spin > (1u << 24) || load_agent(a.flags) & kFlagDevice) {
        atomicOr(a.flags, kFlagDevice);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    s_ok = ok;
  }
  block_sync();
  __threadfence();  // and acquires the other workgroups' writes
  return s_ok != 0;
}

__global__ __launch_bounds__(NT) void g_mid(GArgs a) {
  __shared__ MidShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || pl->nscatter <= 2) return;
  const int S = (int)pl->nscatter;
  const int G = a.mid.blocks;
  uint32_t gen = 0;
  for (int s = 1; s < S - 1; ++s) {
    if ((int)blockIdx.x < G) count_block(a, s, blockIdx.x, a.mid, false, sh.count, NT);
    if (!grid_barrier(a, ++gen)) return;
    for (int b = blockIdx.x; b < (int)pl->nbins[s]; b += gridDim.x)
      column_scan<NT>(a, s, b, false, G, sh.scan.scan32, sh.scan.scan64);
    if (!grid_barrier(a, ++gen)) return;
    if ((int)blockIdx.x < G) scatter_block<false>(a, s, blockIdx.x, a.mid, sh.scatter);
    if (!grid_barrier(a, ++gen)) return;
  }
}

// ---- final pass --------------------------------------------------------------
struct FinalShared {
  uint64_t stage[T];
  uint32_t excl[kMaxBins + 1];  // tile digit offsets, then position bases
  uint64_t wsum[kMaxBins];      // tile digit length sums, then wait bases
  uint64_t clo[256];
  uint64_t chi[256];
  uint64_t scan64[NW + 1];
  uint32_t scan32[NW + 1];
};

template <typename unused = void>
__global__ __launch_bounds__(NT, kScatterWavesPerSimd) void g_final(GArgs a) {
  __shared__ FinalShared sh;
  uint16_t* cnt = reinterpret_cast<uint16_t*>(sh.stage);
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
  const int g = blockIdx.x;
  const int s = (int)pl->nscatter - 1;
  const int nb = (int)pl->nbins[s];
  const int nbits = (int)pl->nbits[s];
  const uint32_t dshift = pl->shift[s];
  const uint32_t dmask = (1u << nbits) - 1;
  KeyCodec kc;
  kc.init(a, pl);
  const bool packed = pl->packed != 0;
  const uint64_t* keys_in = a.keys[(s - 1) & 1];
  const uint32_t* ids_in = a.ids[(s - 1) & 1];
  auto digit_of = [&](uint64_t k) { return (kc.u2(k) >> dshift) & dmask; };

  for (int b = t; b < kMaxBins; b += NT) sh.wsum[b] = 0;
  for (int b = t; b < 256; b += NT) sh.clo[b] = sh.chi[b] = 0;
  // running position and wait offsets of this thread's digits
  uint32_t carry_c[BPT];
  start_offsets(a, s, nb, g, carry_c, sh.scan32);
  uint64_t carry_w[BPT];
  {
    uint64_t wv[BPT];
    uint64_t sum = 0;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int b = t * BPT + i;
      wv[i] = b < nb ? a.hist_w[b] : 0ull;
      sum += wv[i];
    }
    uint64_t tot;
    uint64_t ex = block_excl_scan_u64<NT>(sum, sh.scan64, tot);
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int b = t * BPT + i;
      carry_w[i] = ex + (b < nb ? a.block_histw[(size_t)g * kMaxBins + b] : 0ull);
      ex += wv[i];
    }
  }

  const int tile0 = g * a.main.tpb;
  const int tile1 = min(a.tiles, tile0 + a.main.tpb);
  for (int tile = tile0; tile < tile1; ++tile) {
    block_sync();
    const int64_t tb = (int64_t)tile * T;
    const int cv = (int)min((int64_t)T, a.n - tb);
    const int wb = w * kWave * K;

    // ---- load, digit, per-digit length sums, stable rank, stage ---------
    uint32_t js[K];
    {
      uint64_t key[K];
      uint32_t id[K], dg[K], rk[K];
#pragma unroll
      for (int r = 0; r < K; ++r) {
        const int il = wb + r * kWave + lane;
        key[r] = 0;
        id[r] = 0;
        js[r] = 0;
        dg[r] = (uint32_t)nb - 1;
        if (il < cv) {
          const int64_t i = tb + il;
          if (packed) {
            const uint64_t e = keys_in[i];
            key[r] = e >> kc.W;
            id[r] = (uint32_t)(e & kc.idmask);
          } else {
            key[r] = keys_in[i];
            id[r] = ids_in[i];
          }
          dg[r] = digit_of(key[r]);
          atomicAdd((unsigned long long*)&sh.wsum[dg[r]], (unsigned long long)kc.len(key[r]));
        }
      }
      rank_tile(dg, rk, nb, nbits, cnt, sh.excl, sh.scan32);
      block_sync();  // counters read before the stage is reused
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
      for (int r = 0; r < K; ++r) sh.stage[rk[r]] = packed ? ((key[r] << kc.W) | id[r]) : key[r];
    }

    // ---- per-digit position and wait bases of this tile -------------------
    {
      uint32_t e0[BPT], cagg[BPT];
      uint64_t wagg[BPT];
      uint64_t wloc = 0;
#pragma unroll
      for (int i = 0; i < BPT; ++i) {
        const int b = t * BPT + i;
        e0[i] = b < nb ? sh.excl[b] : 0u;
        cagg[i] = b < nb ? sh.excl[b + 1] - sh.excl[b] : 0u;
        wagg[i] = b < nb ? sh.wsum[b] : 0ull;
        wloc += wagg[i];
      }
      // tile-local length prefix at the start of each of this thread's digits;
      // the scan's barriers also order the reads above before the writes below
      uint64_t wtot;
      uint64_t wfirst = block_excl_scan_u64<NT>(wloc, sh.scan64, wtot);
#pragma unroll
      for (int i = 0; i < BPT; ++i) {
        const int b = t * BPT + i;
        if (b < nb) {
          sh.excl[b] = carry_c[i] - e0[i];    // position base of digit b
          sh.wsum[b] = carry_w[i] - wfirst;   // wait base of digit b
        }
        wfirst += wagg[i];
        carry_c[i] += cagg[i];
        carry_w[i] += wagg[i];
      }
    }
    block_sync();

    // ---- waits: exclusive length prefix over the tile's sorted order ----
    uint64_t el[K];
    uint64_t wsum = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      el[r] = j < cv ? sh.stage[j] : 0ull;
      if (j < cv) wsum += kc.len(packed ? (el[r] >> kc.W) : el[r]);
    }
    uint64_t wtot = wave_incl_scan_u64(wsum);
    wtot = last_lane_u64(wtot);
    uint64_t dummy;
    uint64_t run = block_excl_scan_u64<NT>(lane == 0 ? wtot : 0, sh.scan64, dummy);
    run = __shfl(run, 0, kWave);
    int cur = -1;
    U128 acc = {0, 0};
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      const bool valid = j < cv;
      const uint64_t key = packed ? (el[r] >> kc.W) : el[r];
      const uint32_t ls = valid ? kc.len(key) : 0u;
      const uint64_t incl = wave_incl_scan_len(ls);
      const uint64_t ex = run + incl - ls;
      run += last_lane_u64(incl);
      if (valid) {
        const uint32_t d = digit_of(key);
        const uint32_t pos = sh.excl[d] + (uint32_t)j;
        const uint64_t wt = sh.wsum[d] + ex;
        if (pos < (uint64_t)a.n) {  // always true for consistent counts
          a.wait[pos] = (int64_t)wt;
          a.order[pos] = (int32_t)(packed ? (uint32_t)(el[r] & kc.idmask) : js[r]);
        }
        const int cls = (int)(kc.pp(key) + kc.pmin);
        if (cls != cur) {
          if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
          cur = cls;
          acc.lo = acc.hi = 0;
        }
        add128(acc, wt);
      }
    }
    if (cur >= 0 && (acc.lo | acc.hi)) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
    block_sync();
    // the per-digit sums are accumulated afresh by the next tile
    for (int b = t; b < nb; b += NT) sh.wsum[b] = 0;
  }

  block_sync();
  for (int c = t; c < a.num_classes; c += NT) {
    U128 v = {sh.clo[c], sh.chi[c]};
    if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + c), a.totals + 2 * (1 + c) + 1, v);
  }
  if (t == 0) {
    U128 gsum = {0, 0};
    for (int c = 0; c < 256; ++c) {
      U128 v = {sh.clo[c], sh.chi[c]};
      add128(gsum, v);
    }
    if (gsum.lo | gsum.hi) atomic_add128(a.totals, a.totals + 1, gsum);
  }
}

__global__ void g_fill_zero(uint32_t* p, size_t count) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = 0;
}

int resident_blocks(const void* kernel, int threads) {
  int dev = 0, cus = 256, occ = 1;
  if (hipGetDevice(&dev) == hipSuccess) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) cus = prop.multiProcessorCount;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, 0) != hipSuccess ||
      occ < 1)
    occ = 1;
  return cus * occ;
}

Split make_split(int64_t n, int resident) {
  const int64_t tiles = (n + T - 1) / T;
  int64_t g = resident;
  if (g > kMaxBlocks) g = kMaxBlocks;
  if (g > tiles) g = tiles;
  if (g < 1) g = 1;
  Split s;
  s.tpb = (int32_t)((tiles + g - 1) / g);
  s.blocks = (int32_t)((tiles + s.tpb - 1) / s.tpb);
  return s;
}

void mark(const StageEvents* ev, int stage, bool after, hipStream_t st) {
  if (!ev) return;
  hipEvent_t e = after ? ev->after[stage] : ev->before[stage];
  if (e) (void)hipEventRecord(e, st);
}

}  // namespace

Split global_split(int64_t n) {
  static const int r = resident_blocks(reinterpret_cast<const void*>(g_final<>), NT);
  return make_split(n, r);
}

Split global_mid_split(int64_t n) {
  static const int r = resident_blocks(reinterpret_cast<const void*>(g_mid), NT);
  return make_split(n, r);
}

hipError_t launch_global_schedule(const GArgs& a, hipStream_t st, const StageEvents* ev) {
  hipLaunchKernelGGL(g_reset, dim3(1), dim3(1024), 0, st, a);
  const int vec_ok = ((uintptr_t)a.priority % 4 == 0) && ((uintptr_t)a.length % 16 == 0);
  const dim3 gm(a.main.blocks);
  mark(ev, 0, false, st);
  hipLaunchKernelGGL(g_hist0, gm, dim3(HT), 0, st, a, vec_ok);
  mark(ev, 0, true, st);
  hipLaunchKernelGGL(g_scan, dim3((1u << a.d0) + 1), dim3(SCT), 0, st, a, 0);
  mark(ev, 1, false, st);
  hipLaunchKernelGGL(g_first<>, gm, dim3(NT), 0, st, a);
  mark(ev, 1, true, st);
  hipLaunchKernelGGL(g_mid, dim3(a.mid.blocks), dim3(NT), 0, st, a);
  hipLaunchKernelGGL(g_histF, gm, dim3(HT), 0, st, a);
  hipLaunchKernelGGL(g_scan, dim3(kMaxBins), dim3(SCT), 0, st, a, 1);
  mark(ev, 2, false, st);
  hipLaunchKernelGGL(g_final<>, gm, dim3(NT), 0, st, a);
  mark(ev, 2, true, st);
  return hipGetLastError();
}

hipError_t launch_fill_zero(uint32_t* p, size_t count, hipStream_t st) {
  if (count == 0) return hipSuccess;
  size_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(g_fill_zero, dim3((unsigned)blocks), dim3(256), 0, st, p, count);
  return hipGetLastError();
}

}  // namespace semsched
