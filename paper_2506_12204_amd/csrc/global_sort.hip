// Multi-pass schedule of one long queue (n > SEM_SEGMENT_CAP).
//
// The schedule is the drained min-heap of Algorithm 1 (MinHeap
// Construction): ids ascending by (priority, length, id). Here it is an LSD
// radix sort over only the live bits of (priority, length), followed by the
// waits of Eq. 1 (the exclusive prefix of service times) and exact per-class
// totals, all fused into the last pass.
//
// Every pass splits the queue into static blocks of consecutive tiles, one
// block per workgroup. A pass first counts the digits of every block, a
// column scan turns the counts into per-block offsets, and the scatter then
// walks its block tile by tile with running per-digit offsets. No workgroup
// ever waits for another inside a kernel, and consecutive tiles of a digit
// land next to each other in memory, written by the same workgroup.
//
//   g_hist0      (its first workgroup also clears the small per-call state
//                and the totals)
//                read (priority, length) once: validate, find the ranges and
//                count the low `d0` bits of every length per block. That
//                digit does not depend on the ranges, so no separate min/max
//                pass is needed.
//   g_scan       per-block digit offsets of one pass (column scans); for the
//                first pass one more workgroup reduces the block ranges into
//                the Plan.
//   g_first      first scatter pass: packs every request into one u64
//                element (key above id) and scatters it by the low length
//                digit, on 16K-item tiles.
//   g_mid        middle passes, only for very wide key ranges: count, scan
//                and scatter by 10-bit digits of u2 = (p - pmin) * H + h, in
//                one launch with bounded grid barriers between the phases
//                (g_mid_count / g_mid_scan / g_mid_scatter: the same as
//                separate launches); it returns at once when two passes
//                suffice.
//   g_histF      counts and length sums of the final digit per block.
//   g_final_big  final scatter for at most 256 final digits on 16K-item
//                tiles; g_final does the same for wider digits on 4K-item
//                tiles, and the general cases. Each request's position and
//                wait come out of the same pass, plus the per-class totals.
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
// Compact final pass: sub-bucket starts of at most this many (bucket, id
// chunk) pairs per block are searched in LDS; blocks spanning more take the
// global-window kernel.
constexpr int kWinCap = 512;
// Requests below this count store through buffer resources (byte offsets of
// the waits stay below 2^31); larger queues take the global-window kernel.
constexpr int64_t kBufferStoreItems = 1ll << 28;

// ------------------------------------------------------------------------
// Run by one workgroup of the first histogram pass: no other workgroup of
// that pass touches this state (a block's range error goes into its block
// ranges, and the plan writer raises the flag).
template <int THREADS>
__device__ void reset_call_state(const GArgs& a) {
  const int t = threadIdx.x;
  if (t == 0) {
    a.flags[0] = 0;
    a.plan->ok = 0;
    a.plan->pay = 0;
    a.plan->pay_shift = 32;
  }
  for (int i = t; i < kMaxScatter * kMaxBins; i += THREADS) a.hist_cnt[i] = 0;
  for (int i = t; i < kMaxBins; i += THREADS) a.hist_w[i] = 0;
  for (int i = t; i < 2 * (1 + a.num_classes); i += THREADS) a.totals[i] = 0;
  if (t == 0) {
    a.msync->arrive = 0;
    a.msync->release = 0;
  }
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

// Items [lo, hi) counted by histogram row `row` of split `sp`: block
// row / rows, its (row % rows)-th share of whole tiles (tpb is a multiple of
// rows).
__device__ __forceinline__ void row_range(const GArgs& a, const Split& sp, int row, int rows,
                                          int64_t& lo, int64_t& hi) {
  const int share = sp.tpb / rows;
  lo = ((int64_t)(row / rows) * sp.tpb + (int64_t)(row % rows) * share) * T;
  hi = min(a.n, lo + (int64_t)share * T);
  lo = min(lo, a.n);
}

// Reduce the block ranges and turn them into the Plan (one workgroup).
__device__ void write_plan(const GArgs& a, int G) {
  __shared__ uint32_t s_red[4][SCT_WAVES];
  uint32_t pl_ = 0xffu, ph = 0, ll = 0xffffffffu, lh = 0;
  for (int g = threadIdx.x; g < G; g += SCT) {
    const uint32_t* r = a.block_ranges + 4 * (size_t)g;
    pl_ = min(pl_, r[0]);
    ph = max(ph, r[1]);  // bit 31: the block found a range error
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
  if (gpmax >> 31) atomicOr(a.flags, kFlagRange);
  if ((gpmax >> 31) || load_agent(a.flags) != 0) {
    pl->ok = 0;
    return;
  }
  const uint32_t d0 = (uint32_t)a.d0;
  const uint32_t P = gpmax - gpmin + 1;
  const uint32_t hmin = glmin >> d0;
  const uint32_t H = (glmax >> d0) - hmin + 1;
  const uint32_t wp = bit_width32(P - 1);
  const uint32_t wh = bit_width32(H - 1);
  const uint32_t wid = bit_width32((uint32_t)(a.n - 1));
  const uint32_t kb = wp + wh + d0;  // live key bits
  pl->pmin = gpmin;
  pl->P = P;
  pl->hmin = hmin;
  pl->H = H;
  pl->wp = wp;
  pl->wh = wh;
  // A key of at most 32 bits sits in the high word above a 32-bit id, so no
  // shifts across words are needed to take an element apart.
  pl->W = (!a.force_wide && kb <= 32) ? 32u : wid;
  pl->packed = (!a.force_wide && kb + pl->W <= 64) ? 1u : 0u;
  pl->small = glmax < (1u << 26) ? 1u : 0u;
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
  // compact layout: two passes, at most 256 final digits (the big-tile final
  // pass), lengths below 2^26, and the sub-bucket starts were counted
  pl->compact = (a.chunked && !a.force_wide && mids == 0 && fb <= 256 && pl->small) ? 1u : 0u;
  // carried ranks: above the final digit's bits, if they fit the u32 element
  pl->pay = 0;
  pl->pay_shift = 32;
  if (pl->compact && a.payload) {
    const uint32_t at = kChunkBits + bit_width32(fb - 1);
    if (at + bit_width32(*a.pay_pmax) <= 32) {
      pl->pay = 1;
      pl->pay_shift = at;
    }
  }
  pl->ok = 1;
}

__global__ __launch_bounds__(HT) void g_hist0(GArgs a, int vec_ok) {
  constexpr int HW = HT / kWave;
  __shared__ uint32_t s_hist[kMaxBins];
  __shared__ uint32_t s_part[kMaxBins];
  __shared__ uint32_t s_red[4][HW];
  const int t = threadIdx.x;
  const int g = blockIdx.x;
  const int nb = 1 << a.d0;
  const uint32_t mask = (uint32_t)nb - 1;

  if (g == 0) reset_call_state<HT>(a);
  int64_t lo, hi;
  row_range(a, a.main, g, kHistRows, lo, hi);
  // The first chunk boundary at or after lo, if it lies in this row: the
  // row also counts the first digits of its ids below it (none when the
  // boundary is lo itself). A row is never longer than a chunk, so it holds
  // at most one boundary.
  int64_t bnd = -1;
  if (a.chunked && hi > lo) {
    const int64_t c = ((lo + (1ll << kChunkBits) - 1) >> kChunkBits) << kChunkBits;
    if (c > 0 && c < hi) bnd = c;
  }
  for (int b = t; b < nb; b += HT) {
    s_hist[b] = 0;
    s_part[b] = 0;
  }
  block_sync();

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
          // the boundary is a multiple of 4: a quad is below it or not
          if (4 * (q + (int64_t)u * HT) < bnd) {
            atomicAdd(&s_part[(uint32_t)lv[u].x & mask], 1u);
            atomicAdd(&s_part[(uint32_t)lv[u].y & mask], 1u);
            atomicAdd(&s_part[(uint32_t)lv[u].z & mask], 1u);
            atomicAdd(&s_part[(uint32_t)lv[u].w & mask], 1u);
          }
        }
      }
    }
    scalar_from = q1 * 4;
  }
  for (int64_t i = scalar_from + t; i < hi; i += HT) {
    const int32_t l = a.length[i];
    rg.add(a.priority[i], l, a.num_classes, mask, s_hist);
    if (i < bnd) atomicAdd(&s_part[(uint32_t)l & mask], 1u);
  }

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
    uint32_t* r = a.block_ranges + 4 * (size_t)g;
    r[0] = pl;  // an empty block leaves the neutral values
    r[1] = ph | (bb << 31);
    r[2] = bl;
    r[3] = bh;
  }
  for (int b = t; b < nb; b += HT) a.block_hist[(size_t)g * kMaxBins + b] = s_hist[b];
  // (a request with a range error makes the whole call fail, so counting it
  // in s_part does not matter)
  if (bnd >= 0) {
    uint32_t* part = a.chunk_part + (size_t)(bnd >> kChunkBits) * kMaxBins;
    for (int b = t; b < nb; b += HT) part[b] = s_part[b];
  }
}

// ------------------------------------------------------------------------
// Column scans: block_hist[g][b] becomes the count of digit b in blocks
// before g (block_histw likewise for length sums); the totals go to
// hist_cnt[s][b] (and hist_w[b]).

// With `chunks` (first digit of the compact layout), column b also yields
// the starts of its sub-buckets relative to the bucket's start:
// sub_start[b][k] = number of ids below k * 2^kChunkBits with first digit b =
// the column prefix at the row holding that boundary + the row's own count
// below it (chunk_part). Entry 0 is 0; entries K .. Kp-1 hold the bucket size.
template <int THREADS>
__device__ void column_scan(const GArgs& a, int s, int b, bool weights, int G,
                            uint32_t* scan32, uint64_t* scan64, bool chunks = false) {
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
  const int64_t row_items = (int64_t)(a.main.tpb / kHistRows) * T;
  uint32_t* sub = a.sub_start + ((size_t)b << a.kpb);
#pragma unroll
  for (int i = 0; i < SCPER; ++i) {
    const int g = g0 + i;
    if (i < per && g < G) {
      a.block_hist[(size_t)g * kMaxBins + b] = run;
      if (chunks) {
        const int64_t lo = (int64_t)g * row_items;
        const int64_t c = ((lo + (1ll << kChunkBits) - 1) >> kChunkBits) << kChunkBits;
        if (c > 0 && c < min(a.n, lo + row_items)) {
          const int k = (int)(c >> kChunkBits);
          sub[k] = run + a.chunk_part[(size_t)k * kMaxBins + b];
        }
      }
    }
    run += v[i];
  }
  if (threadIdx.x == 0) {
    a.hist_cnt[s * kMaxBins + b] = total;
    if (chunks) {
      sub[0] = 0;
      for (int k = a.kchunks; k < (1 << a.kpb); ++k) sub[k] = total;
    }
  }
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
// Whether any block of the compact final pass needs the global-window
// kernel: its positions span more (first-digit bucket, id chunk) pairs than
// the LDS window holds, or the queue is too long for buffer-resource stores.
// One workgroup; the bucket starts are the exclusive scan of the first
// digit's counts. The kernels that return at once for the other kind of
// block then return before their set-up.
__device__ void window_check(const GArgs& a, Plan* pl, uint32_t* scan32) {
  __shared__ uint32_t bstart[kMaxBins + 1];
  __shared__ uint32_t any;
  constexpr int PER = kMaxBins / SCT;
  const int nd = 1 << a.d0;
  uint32_t c[PER];
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = threadIdx.x * PER + i;
    c[i] = d < nd ? a.hist_cnt[d] : 0u;
    sum += c[i];
  }
  if (threadIdx.x == 0) any = a.n >= kBufferStoreItems ? 1u : 0u;
  uint32_t tot;
  uint32_t ex = block_excl_scan_u32<SCT>(sum, scan32, tot);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = threadIdx.x * PER + i;
    if (d <= nd) bstart[d] = ex;
    ex += c[i];
  }
  block_sync();
  auto bucket = [&](uint32_t pos) {  // last d < nd with bstart[d] <= pos
    int lo = 0, hi = nd - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (bstart[mid] <= pos) lo = mid; else hi = mid - 1;
    }
    return lo;
  };
  for (int g = threadIdx.x; g < a.fin.blocks; g += SCT) {
    const int64_t lo = (int64_t)g * a.fin.tpb * T;
    const int64_t hi = min(a.n, lo + (int64_t)a.fin.tpb * T);
    if (hi <= lo) continue;
    const int wn = (bucket((uint32_t)(hi - 1)) - bucket((uint32_t)lo) + 1) << a.kpb;
    if (wn > kWinCap) any = 1u;
  }
  block_sync();
  if (threadIdx.x == 0) pl->cglb = any;
}

__global__ __launch_bounds__(SCT) void g_scan(GArgs a, int final) {
  __shared__ uint32_t scan32[SCT / kWave + 1];
  __shared__ uint64_t scan64[SCT / kWave + 1];
  const int b = blockIdx.x;
  if (!final) {
    if (b == (1 << a.d0)) {
      write_plan(a, a.main.blocks * kHistRows);
      return;
    }
    column_scan<SCT>(a, 0, b, false, a.main.blocks * kHistRows, scan32, scan64,
                     a.chunked != 0);
    return;
  }
  Plan* pl = a.plan;
  if (!pl->ok) return;
  if (b == kMaxBins) {
    if (pl->compact) window_check(a, pl, scan32);
    return;
  }
  const int s = (int)pl->nscatter - 1;
  if (b >= (int)pl->nbins[s]) return;
  column_scan<SCT>(a, s, b, true, a.fin.blocks * kHistRows, scan32, scan64);
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
// the number of the tile's items with digit < b. NB: bits matched (every
// digit is below 2^NB).
template <int NB = 10>
__device__ __forceinline__ void rank_tile(const uint32_t (&dg)[K], uint32_t (&rk)[K],
                                          int nb, int nbits, uint16_t* cnt, uint32_t* excl,
                                          uint32_t* scan32) {
  const int w = threadIdx.x / kWave;
  for (int b = lane_id(); b < nb; b += kWave) cnt[w * kMaxBins + b] = 0;
#pragma unroll
  for (int r = 0; r < K; ++r) rk[r] = rank_round_c<NB>(dg[r], cnt + w * kMaxBins);
  block_sync();
  block_digit_offsets<NT>(cnt, kMaxBins, nb, excl, scan32);
#pragma unroll
  for (int r = 0; r < K; ++r) rk[r] += excl[dg[r]] + cnt[w * kMaxBins + dg[r]];
}

// Global digit bases of pass s (exclusive scan of its digit totals) plus this
// block's offset, for this thread's BPT bins.
__device__ __forceinline__ void start_offsets(const GArgs& a, int s, int nb, int row0,
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
    carry[i] = ex + (b < nb ? a.block_hist[(size_t)row0 * kMaxBins + b] : 0u);
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
    u32_alias* sid = reinterpret_cast<u32_alias*>(stage);
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
  u16_alias* cnt = reinterpret_cast<u16_alias*>(sh.stage);
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
  start_offsets(a, s, nb, FIRST ? g * kHistRows : g, carry, sh.scan32);
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

// ---- fast first pass --------------------------------------------------------
// Keys of at most 32 bits (the element's high word), a first digit of D0 bits
// known at compile time. The pass works on big tiles of kFirstTiles tiles
// (16384 items, one workgroup per CU, a 128 KB stage): with up to 1024
// digits a big tile still writes runs of about 16 consecutive elements per
// digit, so the scattered writes mostly fill whole cache lines. Per big tile:
// rank the R1 rounds of every wave against the wave's own counters, turn the
// counters into tile offsets (owners of the digits scan them across the waves
// and the block), stage the tile in digit order and write it out at the
// running digit offsets. Four barriers per big tile; the next tile's inputs
// are loaded while this one is offset, staged and written.

constexpr int R1 = K * kFirstTiles;  // rounds per thread of a big tile
constexpr int T1 = NT * R1;          // items of a big tile

template <int D0>
struct FirstFastShared {
  uint64_t stage[T1];
  uint16_t cnt[NW][1 << D0];  // wave counters, then the waves' tile offsets
  uint32_t base[1 << D0];     // output position of the tile's first item of a digit
  uint32_t part[NW + 1];      // wave totals of the block scans
};

// Index of this thread's wave, as a value the compiler knows to be uniform
// (so that per-wave bases live in scalar registers and per-round addresses
// are immediate offsets from one lane offset).
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Buffer resource over `bytes` bytes at `base` (raw, untyped). Loads through
// it return 0 past the end instead of touching memory there.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000 /* 32-bit data format, gfx9 */);
}

// Cache policy of loads that stream through data read once: the non-temporal
// bit, so that these lines are the first the L2 evicts and the partly written
// output lines of the scatter stay until their runs complete.
constexpr int kLoadStream = 2;

// Inputs of one big tile of `cnt` items starting at item tb, round-major per
// wave (round r of wave w holds items w*64*R1 + r*64 + lane). Items past the
// tile's end read as zero.
__device__ __forceinline__ void load_first(const GArgs& a, const uint8_t* pri, int64_t tb, int cnt,
                                           uint32_t (&pv)[R1], uint32_t (&lv)[R1]) {
  const int wb = wave_id() * kWave * R1;
  // items of this wave's share (uniform; stated so the descriptor stays scalar)
  const int lim = __builtin_amdgcn_readfirstlane(max(0, min(cnt - wb, kWave * R1)));
  const __amdgpu_buffer_rsrc_t rp = raw_rsrc(pri + tb + wb, (uint32_t)lim);
  const __amdgpu_buffer_rsrc_t rl = raw_rsrc(a.length + tb + wb, (uint32_t)lim * 4u);
  const int lane = lane_id();
#pragma unroll
  for (int r = 0; r < R1; ++r) {
    // the whole offset goes in the vector operand: only that part (with the
    // immediate) is range-checked, the scalar offset is not
    pv[r] = __builtin_amdgcn_raw_buffer_load_b8(rp, lane + r * kWave, 0, kLoadStream);
    lv[r] = __builtin_amdgcn_raw_buffer_load_b32(rl, (lane + r * kWave) * 4, 0, kLoadStream);
  }
}

// Clears this wave's NBIN u16 counters.
template <int NBIN>
__device__ __forceinline__ void clear_wave_counters(uint16_t* cnt) {
  static_assert(NBIN % (kWave * 4) == 0, "whole u64 words per lane");
  u64_alias* c64 = reinterpret_cast<u64_alias*>(cnt);
#pragma unroll
  for (int i = 0; i < NBIN / (kWave * 4); ++i) c64[i * kWave + lane_id()] = 0;
}

// COMPACT: the element written is the compact u32 (final digit u2 above the
// low kChunkBits bits of the id); the key ranked and staged is then
// u2 << D0 | first digit instead of the packed key.
// PAY (compact only): the ordering ranks are all zero (u2 = h) and the
// caller's ranks (GArgs::payload) ride along: bits 24 and up of the staged
// key, then bits pay_shift and up of the element.
template <int D0, bool COMPACT, bool PAY>
__device__ void first_fast(const GArgs& a, int g, FirstFastShared<D0>& sh) {
  constexpr int NBIN = 1 << D0;
  constexpr uint32_t M0 = NBIN - 1;
  constexpr int OWN = NBIN > NT ? NBIN / NT : 1;  // digits per owning thread
  constexpr int OWNERS = NBIN / OWN;
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = wave_id();
  const int wb = w * kWave * R1;
  const bool owner = t < OWNERS;
  const Plan* pl = a.plan;
  const uint32_t pmin = pl->pmin;
  const uint32_t psh = pl->wh + D0;
  const uint32_t hoff = pl->hmin << D0;
  const uint32_t H = pl->H;
  const uint32_t pay_shift = pl->pay_shift;
  const uint8_t* pri = PAY ? a.payload : a.priority;
  uint64_t* out = a.keys[0];
  uint32_t* out32 = reinterpret_cast<uint32_t*>(a.keys[0]);
  uint16_t* mycnt = sh.cnt[w];
  clear_wave_counters<NBIN>(mycnt);

  // running output offset of each owned digit: its global base plus the
  // counts of the blocks before this one
  uint32_t carry[OWN];
  {
    uint32_t c[OWN];
    uint32_t sum = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      c[i] = owner ? a.hist_cnt[t * OWN + i] : 0u;
      sum += c[i];
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan_u32<NT>(sum, sh.part, tot);
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      carry[i] = ex + (owner ? a.block_hist[(size_t)g * kHistRows * kMaxBins + t * OWN + i] : 0u);
      ex += c[i];
    }
  }

  // this block's items: tiles [g * tpb, (g + 1) * tpb), tpb a multiple of kFirstTiles
  const int64_t lo = (int64_t)g * a.main.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)a.main.tpb * T);
  // The loop is rotated: the ranking of tile t + 1 runs at the end of
  // iteration t, after the prefetch of its inputs and the (unconditional,
  // exactly counted) stores of tile t, so that the compiler's waits before
  // the ranking cover the loads only and the stores drain meanwhile.
  uint32_t pv[R1], lv[R1];
  uint32_t key[R1], rk[R1];
  auto tile_items = [&](int64_t tb) { return (int)min((int64_t)T1, hi - tb); };
  // key = (p - pmin) << (wh + d0) | ((l >> d0) - hmin) << d0 | (l & M0), or
  // for COMPACT u2 << d0 | (l & M0) with u2 = (p - pmin) * H + (l >> d0) - hmin;
  // either way its low D0 bits are the digit
  // the ranking's lane masks live in this wave's slice of the stage, which
  // only this wave reads after staging and is done with when it ranks
  // S32 (compact, no carried ranks): the staged item is one u32, u2 << 24 |
  // first digit << 14 | index in the tile (u2 < 256, D0 <= 10, tiles of 2^14),
  // in the first half of the stage; the wave's mask table is then its share of
  // that half.
  constexpr bool S32 = COMPACT && !PAY;
  static_assert(!S32 || (D0 <= 10 && T1 <= (1 << 14)), "staged item fits 32 bits");
  u32_alias* stage32 = reinterpret_cast<u32_alias*>(sh.stage);
  u64_alias* masks = S32 ? reinterpret_cast<u64_alias*>(stage32 + wb)
                         : reinterpret_cast<u64_alias*>(sh.stage + wb);
  auto rank_tile = [&](int cv) {
    clear_wave_masks<NBIN>(masks);
#pragma unroll
    for (int r = 0; r < R1; ++r)
      key[r] = PAY ? ((pv[r] << 24) | (lv[r] - hoff))  // (u2 << D0 < 2^18)
                   : (COMPACT ? (__umul24(pv[r] - pmin, H) << D0) : ((pv[r] - pmin) << psh)) +
                         (lv[r] - hoff);
    if (cv < T1) {
      // items past the end take the last digit: they rank after every real
      // item of it, i.e. at the tile positions >= cv, which are not written
#pragma unroll
      for (int r = 0; r < R1; ++r)
        if (wb + r * kWave + lane >= cv) key[r] |= M0;
    }
#pragma unroll
    for (int r = 0; r < R1; ++r) rk[r] = rank_round_mask(key[r] & M0, masks, mycnt);
  };

  load_first(a, pri, lo, tile_items(lo), pv, lv);
  rank_tile(tile_items(lo));
  for (int64_t tb = lo; tb < hi; tb += T1) {
    const int cv = tile_items(tb);
    const bool more = tb + T1 < hi;
    // the next tile's inputs load while this one is offset, staged and written
    if (more) load_first(a, pri, tb + T1, tile_items(tb + T1), pv, lv);
    block_sync();  // every wave's counters are complete

    uint32_t cw[OWN][NW], tot[OWN];
    uint32_t local = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      tot[i] = 0;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        cw[i][v] = owner ? sh.cnt[v][t * OWN + i] : 0u;
        tot[i] += cw[i][v];
      }
      local += tot[i];
    }
    const uint32_t incl = wave_incl_scan_u32(local);
    if (lane == kWave - 1) sh.part[w] = incl;
    block_sync();
    uint32_t ex = incl - local;
    for (int v = 0; v < w; ++v) ex += sh.part[v];  // (w is uniform)
    if (owner) {
#pragma unroll
      for (int i = 0; i < OWN; ++i) {
        const int b = t * OWN + i;
        uint32_t run = ex;
#pragma unroll
        for (int v = 0; v < NW; ++v) {
          sh.cnt[v][b] = (uint16_t)run;
          run += cw[i][v];
        }
        sh.base[b] = carry[i] - ex;
        carry[i] += tot[i];
        ex += tot[i];
      }
    }
    block_sync();  // tile offsets and bases are written

#pragma unroll
    for (int r = 0; r < R1; ++r) rk[r] += mycnt[opaque(key[r]) & M0];
    clear_wave_counters<NBIN>(mycnt);  // only this wave reads them until the next ranking
    if constexpr (S32) {
#pragma unroll
      for (int r = 0; r < R1; ++r)
        stage32[rk[r]] = ((key[r] >> D0) << 24) | ((key[r] & M0) << 14) |
                         (uint32_t)(wb + r * kWave + lane);
    } else {
#pragma unroll
      for (int r = 0; r < R1; ++r)
        sh.stage[rk[r]] = ((uint64_t)key[r] << 32) | (uint32_t)(tb + wb + r * kWave + lane);
    }
    block_sync();  // the tile is staged in digit order

    // stores are unconditional: lanes without an item write to the sink
    const bool full = cv == T1;
#pragma unroll
    for (int r = 0; r < R1; ++r) {
      const int j = wb + r * kWave + lane;
      if constexpr (S32) {
        const uint32_t e = stage32[j];
        const uint32_t pos = sh.base[(e >> 14) & M0] + (uint32_t)j;
        const bool item = (full || j < cv) && pos < (uint64_t)a.n;
        uint32_t* po = item ? out32 + pos : reinterpret_cast<uint32_t*>(a.sink);
        *po = ((e >> 24) << kChunkBits) |
              ((uint32_t)(tb + (e & 0x3fffu)) & ((1u << kChunkBits) - 1));
        if (r % 8 == 7) __builtin_amdgcn_sched_barrier(0);
        continue;
      }
      const uint64_t e = sh.stage[j];
      const uint32_t pos = sh.base[(uint32_t)(e >> 32) & M0] + (uint32_t)j;
      const bool item = (full || j < cv) && pos < (uint64_t)a.n;  // (pos < n for consistent counts)
      if (COMPACT) {  // u2 above the id's low bits (and the carried rank above u2)
        uint32_t* po = item ? out32 + pos : reinterpret_cast<uint32_t*>(a.sink);
        const uint32_t hi = (uint32_t)(e >> 32);
        const uint32_t u2 = PAY ? (hi & 0xffffffu) >> D0 : hi >> D0;
        const uint32_t rank_bits = PAY ? (hi >> 24) << pay_shift : 0u;
        *po = rank_bits | (u2 << kChunkBits) | ((uint32_t)e & ((1u << kChunkBits) - 1));
      } else {
        uint64_t* po = item ? out + pos : a.sink;
        *po = e;
      }
      // keep the scheduler from hoisting every round's loads at once, which
      // would hold ~5 registers per round live
      if (r % 8 == 7) __builtin_amdgcn_sched_barrier(0);
    }
    if (more) rank_tile(tile_items(tb + T1));
  }
}

// 4 waves per SIMD: two 8-wave workgroups per CU, so one can compute while
// the other waits on memory.
constexpr int kScatterWavesPerSimd = 4;

// The first pass's 148 KB of LDS allow one workgroup per CU: 2 waves per SIMD.
template <int D0>
__global__ __launch_bounds__(NT, 2) void g_first(GArgs a) {
  __shared__ union {
    ScatterShared generic;
    FirstFastShared<D0> fast;
  } sh;
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  if (pl->compact && pl->pay)
    first_fast<D0, true, true>(a, blockIdx.x, sh.fast);
  else if (pl->compact)
    first_fast<D0, true, false>(a, blockIdx.x, sh.fast);
  else if (pl->packed && pl->W == 32)
    first_fast<D0, false, false>(a, blockIdx.x, sh.fast);
  else
    scatter_block<true>(a, 0, blockIdx.x, a.main, sh.generic);
}

// Per-block digit counts (and length sums) of pass s over its input elements.
struct CountShared {
  uint32_t cnt[kMaxBins];
  uint64_t w[kMaxBins];
};

// (Used for the final digit of the generic layouts; the middle passes count
// with count_mid.) Digits of at most 8 values are counted in registers.
__device__ void count_block(const GArgs& a, int s, int g, Split sp, int rows, bool weights,
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
  int64_t lo, hi;
  row_range(a, sp, g, rows, lo, hi);
  // lo is even (a multiple of the tile), so pairs of elements stay aligned
  const int64_t q0 = lo >> 1, q1 = hi >> 1;
  const ulonglong2* k2 = reinterpret_cast<const ulonglong2*>(keys_in);
  auto add = [&](uint64_t e) {
    const uint64_t key = packed ? (e >> kc.W) : e;
    const uint32_t d = (kc.u2(key) >> dshift) & dmask;
    atomicAdd(&sh.cnt[d], 1u);
    if (weights) atomicAdd((unsigned long long*)&sh.w[d], (unsigned long long)kc.len(key));
  };
  // With few digits every element would hit the same few LDS words: each
  // lane then keeps its own counts and length sums in registers and the wave
  // adds them up once at the end.
  constexpr int kFew = 8;
  uint32_t fc[kFew];
  uint64_t fw[kFew];
  const bool few = nb <= kFew;
#pragma unroll
  for (int b = 0; b < kFew; ++b) {
    fc[b] = 0;
    fw[b] = 0;
  }
  auto add_few = [&](uint64_t e) {
    const uint64_t key = packed ? (e >> kc.W) : e;
    const uint32_t d = (kc.u2(key) >> dshift) & dmask;
    const uint64_t l = weights ? (uint64_t)kc.len(key) : 0;
#pragma unroll
    for (int b = 0; b < kFew; ++b) {
      const bool on = d == (uint32_t)b;
      fc[b] += on ? 1u : 0u;
      fw[b] += on ? l : 0;
    }
  };
  for (int64_t q = q0 + t; q < q1; q += (int64_t)threads * HU) {
    ulonglong2 v[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) v[u] = k2[min(q + (int64_t)u * threads, q1 - 1)];
#pragma unroll
    for (int u = 0; u < HU; ++u) {
      if (q + (int64_t)u * threads < q1) {
        if (few) {
          add_few(v[u].x);
          add_few(v[u].y);
        } else {
          add(v[u].x);
          add(v[u].y);
        }
      }
    }
  }
  if (few) {
#pragma unroll
    for (int b = 0; b < kFew; ++b) {
      if (b < nb) {  // (nb is uniform)
        const uint32_t tc = (uint32_t)__builtin_amdgcn_readlane(
            (int)wave_incl_scan_u32(fc[b]), kWave - 1);
        const uint64_t tw = weights ? last_lane_u64(wave_incl_scan_u64(fw[b])) : 0;
        if (lane_id() == 0) {
          if (tc) atomicAdd(&sh.cnt[b], tc);
          if (tw) atomicAdd((unsigned long long*)&sh.w[b], (unsigned long long)tw);
        }
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

// The big-tile final pass (below) handles final digits of at most 256
// values with keys in the high word, two passes and lengths below 2^26.
__device__ __forceinline__ bool use_big_final(const Plan* pl) {
  return pl->packed && pl->W == 32 && pl->nscatter == 2 && pl->small && pl->nbins[1] <= 256;
}

// Its wide form (in the kernel g_final_cglb, which is launched when the
// queue is chunked) takes the other keys in the high word with at most 256
// final digits: after middle passes or with lengths of 2^26 and more.
__device__ __forceinline__ bool use_wide_big_final(const GArgs& a, const Plan* pl) {
  return a.chunked && pl->packed && pl->W == 32 && !pl->compact && !use_big_final(pl) &&
         pl->nbins[pl->nscatter - 1] <= 256;
}

// Final-digit histogram of one row when the big final pass runs (keys in the
// high word, two passes, at most 256 final digits). Every wave counts into
// bins of its own, so lanes of different waves never meet on an LDS address
// (with few digits that contention dominated), and a bin's count and length
// sum share one u64: the count above bit csh, the lengths below, which the
// caller has checked cannot reach bit csh.
constexpr int kHistFBins = 256;
struct HistFShared {
  uint64_t h[HT / kWave][kHistFBins];
};

__device__ void histF_fast(const GArgs& a, int row, int64_t lo, int64_t hi, uint32_t csh,
                           HistFShared& sh) {
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int w = wave_id();
  const int nb = (int)pl->nbins[1];
  const uint32_t d0 = (uint32_t)a.d0;
  const uint32_t psh = pl->wh + d0;
  const uint32_t H = pl->H;
  const uint32_t mh = (1u << pl->wh) - 1;
  const uint32_t lenmask = (1u << psh) - 1;
  const uint32_t hoff = pl->hmin << d0;
  const uint64_t one = 1ull << csh;
  clear_wave_counters<4 * kHistFBins>(reinterpret_cast<uint16_t*>(sh.h[w]));
  auto add = [&](uint64_t e) {
    const uint32_t key = (uint32_t)(e >> 32);
    const uint32_t d = __umul24(key >> psh, H) + ((key >> d0) & mh);
    atomicAdd((unsigned long long*)&sh.h[w][d], (unsigned long long)(one | ((key & lenmask) + hoff)));
  };
  const uint64_t* keys_in = a.keys[0];
  // lo is even (a multiple of the tile), so pairs of elements stay aligned
  const int64_t q0 = lo >> 1, q1 = hi >> 1;
  const ulonglong2* k2 = reinterpret_cast<const ulonglong2*>(keys_in);
  for (int64_t q = q0 + t; q < q1; q += (int64_t)HT * HU) {
    ulonglong2 v[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) v[u] = k2[min(q + (int64_t)u * HT, q1 - 1)];
#pragma unroll
    for (int u = 0; u < HU; ++u) {
      if (q + (int64_t)u * HT < q1) {
        add(v[u].x);
        add(v[u].y);
      }
    }
  }
  if ((hi & 1) && t == 0 && hi > lo) add(keys_in[hi - 1]);
  block_sync();
  for (int b = t; b < nb; b += HT) {
    uint64_t sum = 0;
#pragma unroll
    for (int v = 0; v < HT / kWave; ++v) sum += sh.h[v][b];
    a.block_hist[(size_t)row * kMaxBins + b] = (uint32_t)(sum >> csh);
    a.block_histw[(size_t)row * kMaxBins + b] = sum & (one - 1);
  }
}

// ---- compact layout: positions -> (first digit, id chunk) ----------------------

// bstart[d] = position of the first element of first-digit bucket d after the
// first pass (exclusive scan of that pass's digit totals), for d < 2^d0, and
// bstart[2^d0] = n. Every thread of the workgroup must call it.
template <int THREADS>
__device__ void bucket_starts(const GArgs& a, uint32_t* bstart, uint32_t* scan32) {
  constexpr int PER = kMaxBins / THREADS;
  const int nd = 1 << a.d0;
  uint32_t c[PER];
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = threadIdx.x * PER + i;
    c[i] = d < nd ? a.hist_cnt[d] : 0u;
    sum += c[i];
  }
  uint32_t tot;
  uint32_t ex = block_excl_scan_u32<THREADS>(sum, scan32, tot);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = threadIdx.x * PER + i;
    if (d <= nd) bstart[d] = ex;  // d == nd: the total
    ex += c[i];
  }
  if (threadIdx.x == 0 && nd == kMaxBins) bstart[nd] = tot;
  block_sync();
}

// Last bucket d < nd with bstart[d] <= pos. Empty buckets share their start
// with the next one, so the bucket found is the one that holds pos.
__device__ __forceinline__ int bucket_of(const uint32_t* bstart, int nd, uint32_t pos) {
  int lo = 0, hi = nd - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (bstart[mid] <= pos) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Class (relative, p - pmin) of final digit u2 = class * H + h: u2 / H by a
// multiply with m = ceil(2^22 / H). Exact for u2 < 1024 and H <= 1024: the
// product exceeds u2 * 2^22 / H by less than u2 / 2^22 < 1/1024 <= 1/H, and
// u2 * m < 2^32.
__device__ __forceinline__ uint32_t div_magic(uint32_t H) {
  return ((1u << 22) + H - 1) / H;
}
__device__ __forceinline__ uint32_t class_of(uint32_t u2, uint32_t magic) {
  return __umul24(u2, magic) >> 22;  // both factors below 2^24
}

// Final-digit histogram of one row for the compact layout: per final digit
// the count and the sum of first digits (the element holds the final digit;
// the first digit is the bucket its position lies in, followed by a cursor,
// since a thread's positions increase). The row's length sum of digit u2 is
// count * (h + hmin) * 2^d0 + that sum.
struct HistFCompactShared {
  uint64_t h[HT / kWave][kHistFBins];
  uint32_t bstart[kMaxBins + 1];
  uint32_t scan32[HT / kWave + 1];
};

__device__ void histF_compact(const GArgs& a, int row, int64_t lo, int64_t hi,
                              HistFCompactShared& sh) {
  // count above bit 36: a row holds fewer than 2^23 elements, so its first
  // digits add up to less than 2^33
  constexpr uint32_t CSH = 36;
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int w = wave_id();
  const int nb = (int)pl->nbins[1];
  const int nd = 1 << a.d0;
  clear_wave_counters<4 * kHistFBins>(reinterpret_cast<uint16_t*>(sh.h[w]));
  bucket_starts<HT>(a, sh.bstart, sh.scan32);  // (ends with a barrier)

  const uint32_t* keys_in = reinterpret_cast<const uint32_t*>(a.keys[0]);
  uint64_t* bins = sh.h[w];
  // lo is a multiple of 4 (of the tile), so quads of elements stay aligned
  const int64_t q0 = lo >> 2, q1 = hi >> 2;
  const uint4* k4 = reinterpret_cast<const uint4*>(keys_in);
  int d = 0;
  uint32_t nxt = 0;  // start of bucket d + 1
  if (q0 + t < q1) {
    d = bucket_of(sh.bstart, nd, (uint32_t)(4 * (q0 + t)));
    nxt = sh.bstart[d + 1];
  }
  const uint32_t dbits = pl->pay_shift - kChunkBits;  // digit bits (carried ranks above)
  auto add = [&](uint32_t e, uint32_t pos) {
    while (pos >= nxt) nxt = sh.bstart[++d + 1];
    atomicAdd((unsigned long long*)&bins[__builtin_amdgcn_ubfe(e, kChunkBits, dbits)],
              (unsigned long long)((1ull << CSH) | (uint32_t)d));
  };
  for (int64_t q = q0 + t; q < q1; q += (int64_t)HT * HU) {
    uint4 v[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) v[u] = k4[min(q + (int64_t)u * HT, q1 - 1)];
#pragma unroll
    for (int u = 0; u < HU; ++u) {
      const int64_t qq = q + (int64_t)u * HT;
      if (qq < q1) {
        const uint32_t p0 = (uint32_t)(4 * qq);
        add(v[u].x, p0);
        add(v[u].y, p0 + 1);
        add(v[u].z, p0 + 2);
        add(v[u].w, p0 + 3);
      }
    }
  }
  // the last (n % 4) elements of the queue
  if (t < (int)(hi - 4 * q1)) {
    const uint32_t pos = (uint32_t)(4 * q1 + t);
    d = bucket_of(sh.bstart, nd, pos);
    nxt = sh.bstart[d + 1];
    add(keys_in[pos], pos);
  }
  block_sync();
  const uint32_t H = pl->H;
  const uint32_t magic = div_magic(H);
  for (int b = t; b < nb; b += HT) {
    uint64_t sum = 0;
#pragma unroll
    for (int v = 0; v < HT / kWave; ++v) sum += sh.h[v][b];
    const uint64_t cnt = sum >> CSH;
    const uint32_t hh = (uint32_t)b - class_of((uint32_t)b, magic) * H;
    a.block_hist[(size_t)row * kMaxBins + b] = (uint32_t)cnt;
    a.block_histw[(size_t)row * kMaxBins + b] =
        cnt * ((uint64_t)(hh + pl->hmin) << a.d0) + (sum & ((1ull << CSH) - 1));
  }
}

__global__ __launch_bounds__(HT) void g_histF(GArgs a) {
  __shared__ union {
    CountShared generic;
    HistFShared fast;
    HistFCompactShared compact;
  } sh;
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  const int row = blockIdx.x;
  if (pl->compact) {
    int64_t lo, hi;
    row_range(a, a.fin, row, kHistRows, lo, hi);
    histF_compact(a, row, lo, hi, sh.compact);
    return;
  }
  if (use_big_final(pl)) {
    int64_t lo, hi;
    row_range(a, a.fin, row, kHistRows, lo, hi);
    // count above csh, lengths below: the row's lengths add up to less than
    // items * (largest length + 1), which must stay below 2^csh
    const uint32_t ib = bit_width32((uint32_t)max((int64_t)1, hi - lo));
    const uint32_t lb = bit_width32(((pl->hmin + pl->H) << a.d0));
    const uint32_t csh = 64 - ib;
    if (ib + lb <= csh) {
      histF_fast(a, row, lo, hi, csh, sh.fast);
      return;
    }
  }
  count_block(a, (int)pl->nscatter - 1, row, a.fin, kHistRows, true, sh.generic, HT);
}

// ---- fast middle pass ---------------------------------------------------------
// Packed u64 elements (key above W id bits) moved by a 10-bit digit of u2,
// with the big tiles, wave counters, owner offsets and rotated loop of the
// fast first pass: a big tile of 16384 items writes runs of about 16
// consecutive elements per digit, against 4 on the 4096-item tiles of the
// generic scatter, so most written lines are whole.
struct MidFastShared {
  uint64_t stage[T1];
  uint16_t cnt[NW][kMaxBins];  // wave counters, then the waves' tile offsets
  uint32_t base[kMaxBins];     // output position of the tile's first item of a digit
  uint32_t part[NW + 1];
};

__device__ void mid_fast(const GArgs& a, int s, int g, MidFastShared& sh) {
  constexpr int NBIN = kMaxBins;
  constexpr uint32_t M = NBIN - 1;
  constexpr int OWN = NBIN / NT;  // digits per owning thread (every thread owns)
  static_assert(OWN * NT == NBIN, "every digit has an owner");
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = wave_id();
  const int wb = w * kWave * R1;
  const Plan* pl = a.plan;
  KeyCodec kc;
  kc.init(a, pl);
  const uint32_t dshift = pl->shift[s];
  const uint64_t* in = a.keys[(s - 1) & 1];
  uint64_t* out = a.keys[s & 1];
  uint16_t* mycnt = sh.cnt[w];
  clear_wave_counters<NBIN>(mycnt);
  auto digit = [&](uint64_t e) { return (kc.u2(e >> kc.W) >> dshift) & M; };

  uint32_t carry[OWN];
  {
    uint32_t c[OWN];
    uint32_t sum = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      c[i] = a.hist_cnt[s * kMaxBins + t * OWN + i];
      sum += c[i];
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan_u32<NT>(sum, sh.part, tot);
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      carry[i] = ex + a.block_hist[(size_t)g * kMaxBins + t * OWN + i];
      ex += c[i];
    }
  }

  const int64_t lo = (int64_t)g * a.mid.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)a.mid.tpb * T);
  uint64_t ev[R1];  // this tile's elements (the digits are recomputed from them)
  uint32_t rk[R1];
  auto tile_items = [&](int64_t tb) { return (int)min((int64_t)T1, hi - tb); };
  // buffer loads over this wave's share of the tile: one scalar base, the
  // lane's offset plus an immediate per round; items past the end read 0
  auto load = [&](int64_t tb, uint64_t (&dst)[R1]) {
    const int lim = __builtin_amdgcn_readfirstlane(
        (int)max((int64_t)0, min(hi - tb - wb, (int64_t)kWave * R1)));
    const __amdgpu_buffer_rsrc_t rs = raw_rsrc(in + tb + wb, (uint32_t)lim * 8u);
#pragma unroll
    for (int r = 0; r < R1; ++r) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, (lane + r * kWave) * 8, 0, 0);
      dst[r] = (uint64_t)v[0] | ((uint64_t)v[1] << 32);
    }
  };
  // items past the end take the last digit and rank after every real one
  auto digit_at = [&](int r, int cv) { return wb + r * kWave + lane < cv ? digit(ev[r]) : M; };
  // lane-mask ranking, the masks in this wave's slice of the stage (as in the
  // first pass)
  u64_alias* masks = reinterpret_cast<u64_alias*>(sh.stage + wb);
  auto rank = [&](int cv) {
    clear_wave_masks<NBIN>(masks);
#pragma unroll
    for (int r = 0; r < R1; ++r) rk[r] = rank_round_mask(digit_at(r, cv), masks, mycnt);
  };

  if (lo < hi) {
    load(lo, ev);
    rank(tile_items(lo));
  }
  for (int64_t tb = lo; tb < hi; tb += T1) {
    const int cv = tile_items(tb);
    const bool more = tb + T1 < hi;
    uint64_t nx[R1];  // the next tile's elements load while this one is offset and written
    if (more) load(tb + T1, nx);
    block_sync();  // every wave's counters are complete

    uint32_t cw[OWN][NW], tot[OWN];
    uint32_t local = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      tot[i] = 0;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        cw[i][v] = sh.cnt[v][t * OWN + i];
        tot[i] += cw[i][v];
      }
      local += tot[i];
    }
    const uint32_t incl = wave_incl_scan_u32(local);
    if (lane == kWave - 1) sh.part[w] = incl;
    block_sync();
    uint32_t ex = incl - local;
    for (int v = 0; v < w; ++v) ex += sh.part[v];  // (w is uniform)
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int b = t * OWN + i;
      uint32_t run = ex;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        sh.cnt[v][b] = (uint16_t)run;
        run += cw[i][v];
      }
      sh.base[b] = carry[i] - ex;
      carry[i] += tot[i];
      ex += tot[i];
    }
    block_sync();  // tile offsets and bases are written

#pragma unroll
    for (int r = 0; r < R1; ++r) rk[r] += mycnt[opaque(digit_at(r, cv))];
    clear_wave_counters<NBIN>(mycnt);  // only this wave reads them until the next ranking
#pragma unroll
    for (int r = 0; r < R1; ++r) sh.stage[rk[r]] = ev[r];
    block_sync();  // the tile is staged in digit order

    const bool full = cv == T1;
#pragma unroll
    for (int r = 0; r < R1; ++r) {
      const int j = wb + r * kWave + lane;
      const uint64_t e = sh.stage[j];
      const uint32_t pos = sh.base[digit(e)] + (uint32_t)j;
      const bool item = (full || j < cv) && pos < (uint64_t)a.n;  // (pos < n for consistent counts)
      uint64_t* po = item ? out + pos : a.sink;
      *po = e;
      if (r % 8 == 7) __builtin_amdgcn_sched_barrier(0);
    }
    if (more) {
#pragma unroll
      for (int r = 0; r < R1; ++r) ev[r] = nx[r];
      rank(tile_items(tb + T1));
    }
  }
}

// ---- middle passes: one launch with grid barriers, or three per pass ----
// Digit counts of one block of a middle pass: every wave counts into a table
// of its own (no LDS atomics between waves), summed at the end.
struct CountMidShared {
  uint32_t cnt[NW][kMaxBins];
};

__device__ void count_mid(const GArgs& a, int s, int g, CountMidShared& sh) {
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int w = t / kWave;
  const uint32_t dshift = pl->shift[s];
  constexpr uint32_t M = kMaxBins - 1;  // middle passes have 1024 digits
  KeyCodec kc;
  kc.init(a, pl);
  const bool packed = pl->packed != 0;
  const uint64_t* keys_in = a.keys[(s - 1) & 1];
  uint32_t* flat = &sh.cnt[0][0];
  for (int i = t; i < NW * kMaxBins; i += NT) flat[i] = 0;
  block_sync();
  int64_t lo, hi;
  row_range(a, a.mid, g, 1, lo, hi);
  uint32_t* mine = sh.cnt[w];
  auto add = [&](uint64_t e) {
    const uint64_t key = packed ? (e >> kc.W) : e;
    atomicAdd(&mine[(kc.u2(key) >> dshift) & M], 1u);
  };
  // lo is even (a multiple of the tile), so pairs of elements stay aligned
  const int64_t q0 = lo >> 1, q1 = hi >> 1;
  const ulonglong2* k2 = reinterpret_cast<const ulonglong2*>(keys_in);
  for (int64_t q = q0 + t; q < q1; q += (int64_t)NT * HU) {
    ulonglong2 v[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) v[u] = k2[min(q + (int64_t)u * NT, q1 - 1)];
#pragma unroll
    for (int u = 0; u < HU; ++u) {
      if (q + (int64_t)u * NT < q1) {
        add(v[u].x);
        add(v[u].y);
      }
    }
  }
  if ((hi & 1) && t == 0 && hi > lo) add(keys_in[hi - 1]);
  block_sync();
  for (int b = t; b < kMaxBins; b += NT) {
    uint32_t c = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) c += sh.cnt[v][b];
    a.block_hist[(size_t)g * kMaxBins + b] = c;
  }
}

// Column scans of four adjacent digits b0 .. b0+3 of a middle pass at once
// (one 16-byte load per block row), as column_scan does for one digit.
__device__ void column_scan4(const GArgs& a, int s, int b0, int G, uint32_t (*part)[4]) {
  constexpr int PER = kMaxBlocks / NT;
  const int per = (G + NT - 1) / NT;
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
  const int g0 = t * per;
  uint4 v[PER];
  uint32_t loc[4] = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    v[i] = make_uint4(0, 0, 0, 0);
    if (i < per && g0 + i < G)
      v[i] = *reinterpret_cast<const uint4*>(a.block_hist + (size_t)(g0 + i) * kMaxBins + b0);
    loc[0] += v[i].x;
    loc[1] += v[i].y;
    loc[2] += v[i].z;
    loc[3] += v[i].w;
  }
  uint32_t run[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t inc = wave_incl_scan_u32(loc[k]);
    run[k] = inc - loc[k];
    if (lane == kWave - 1) part[w][k] = inc;
  }
  block_sync();
  uint32_t total[4] = {0, 0, 0, 0};
#pragma unroll
  for (int u = 0; u < NT / kWave; ++u) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      run[k] += u < w ? part[u][k] : 0u;
      total[k] += part[u][k];
    }
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (i < per && g0 + i < G) {
      *reinterpret_cast<uint4*>(a.block_hist + (size_t)(g0 + i) * kMaxBins + b0) =
          make_uint4(run[0], run[1], run[2], run[3]);
      run[0] += v[i].x;
      run[1] += v[i].y;
      run[2] += v[i].z;
      run[3] += v[i].w;
    }
  }
  if (t < 4) a.hist_cnt[s * kMaxBins + b0 + t] = total[t];
  block_sync();  // part is reused by the next call
}

union MidShared {
  ScatterShared scatter;
  MidFastShared fast;
  CountMidShared count;
  uint32_t part4[NT / kWave][4];
};

// Grid barrier of the middle-pass kernel, a normal launch whose grid is the
// number of workgroups that fit on the device at once. Workgroup leaders add
// to the arrival count; the last to arrive resets it and publishes the
// barrier's generation in the release word, which the others poll. The wait
// is bounded: if the workgroups were not all resident (another program
// holding CUs), a leader gives up after a.mid_spin polls, records
// kFlagDevice, clears the plan's ok word (so the kernels after this one do
// nothing) and every workgroup leaves at its next barrier; the blocking
// calls then run the schedule again with the middle passes as separate
// launches per phase, which need no residency.
__device__ bool grid_barrier(const GArgs& a, uint32_t gen) {
  __shared__ uint32_t s_ok;
  __threadfence();  // release this workgroup's writes at agent scope
  block_sync();
  if (threadIdx.x == 0) {
    uint32_t ok = 1;
    if (atomicAdd(&a.msync->arrive, 1u) == gridDim.x - 1) {
      __hip_atomic_store(&a.msync->arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.msync->release, gen, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      // relaxed polls: an acquire load would invalidate this XCD's L2 at
      // every poll, under the workgroups still working there; the fence
      // after the wait orders what follows
      for (uint32_t spin = 0; __hip_atomic_load(&a.msync->release, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT) < gen;
           ++spin) {
        if (spin >= a.mid_spin || ((spin & 63) == 63 && (load_agent(a.flags) & kFlagDevice))) {
          atomicOr(a.flags, kFlagDevice);
          // the later kernels of this schedule then return at once
          __hip_atomic_store(&a.plan->ok, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ok = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (load_agent(a.flags) & kFlagDevice) ok = 0;
    s_ok = ok;
  }
  block_sync();
  __threadfence();  // acquire the other workgroups' writes
  return s_ok != 0;
}

// The middle passes: per pass, count every block, scan the counts per digit
// over the blocks, scatter every block, with grid barriers between the phases.
__global__ __launch_bounds__(NT) void g_mid(GArgs a) {
  __shared__ MidShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || pl->nscatter <= 2) return;
  const int S = (int)pl->nscatter;
  const int G = a.mid.blocks;
  uint32_t gen = 0;
  for (int s = 1; s < S - 1; ++s) {
    if ((int)blockIdx.x < G) count_mid(a, s, blockIdx.x, sh.count);
    if (!grid_barrier(a, ++gen)) return;
    for (int b = blockIdx.x; b < kMaxBins / 4; b += gridDim.x) column_scan4(a, s, 4 * b, G, sh.part4);
    if (!grid_barrier(a, ++gen)) return;
    if ((int)blockIdx.x < G) {
      if (pl->packed)
        mid_fast(a, s, blockIdx.x, sh.fast);
      else
        scatter_block<false>(a, s, blockIdx.x, a.mid, sh.scatter);
    }
    if (!grid_barrier(a, ++gen)) return;
  }
}

// The same middle pass s as three launches (count, scan, scatter), for a
// schedule run again after the barrier of g_mid gave up. A launch whose pass
// the plan does not need returns at once.
__global__ __launch_bounds__(NT) void g_mid_count(GArgs a, int s) {
  __shared__ MidShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || s >= (int)pl->nscatter - 1) return;
  count_mid(a, s, blockIdx.x, sh.count);
}

__global__ __launch_bounds__(NT) void g_mid_scan(GArgs a, int s) {
  __shared__ uint32_t part4[NT / kWave][4];
  const Plan* pl = a.plan;
  if (!pl->ok || s >= (int)pl->nscatter - 1) return;
  column_scan4(a, s, 4 * blockIdx.x, a.mid.blocks, part4);
}

__global__ __launch_bounds__(NT) void g_mid_scatter(GArgs a, int s) {
  __shared__ MidShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || s >= (int)pl->nscatter - 1) return;
  if (pl->packed)
    mid_fast(a, s, blockIdx.x, sh.fast);
  else
    scatter_block<false>(a, s, blockIdx.x, a.mid, sh.scatter);
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

__device__ void final_generic(const GArgs& a, int g, FinalShared& sh) {
  u16_alias* cnt = reinterpret_cast<u16_alias*>(sh.stage);
  const Plan* pl = a.plan;
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
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
  start_offsets(a, s, nb, g * kHistRows, carry_c, sh.scan32);
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
      carry_w[i] = ex + (b < nb ? a.block_histw[(size_t)g * kHistRows * kMaxBins + b] : 0ull);
      ex += wv[i];
    }
  }

  const int tile0 = g * a.fin.tpb;
  const int tile1 = min(a.tiles, tile0 + a.fin.tpb);
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
      // (few final digits, e.g. after middle passes: match only their bits)
      if (nbits <= 2)
        rank_tile<2>(dg, rk, nb, nbits, cnt, sh.excl, sh.scan32);
      else if (nbits <= 5)
        rank_tile<5>(dg, rk, nb, nbits, cnt, sh.excl, sh.scan32);
      else
        rank_tile<10>(dg, rk, nb, nbits, cnt, sh.excl, sh.scan32);
      block_sync();  // counters read before the stage is reused
      if (!packed) {
        u32_alias* sid = reinterpret_cast<u32_alias*>(sh.stage);
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

// ---- fast final pass ----------------------------------------------------------
// Keys of at most 32 bits, two scatter passes (the final digit is the whole
// mixed-radix value u2 = (p - pmin) * H + h, so a digit holds one class),
// lengths below 2^26. Per tile:
//   phase 1   digit and length of every item; per-digit length sums of the
//             tile (LDS atomics); stable ranks against the wave counters.
//   offsets   owners of the bins scan counts and length sums across waves
//             and the block: tile offsets for the ranks, and for every digit
//             the output position of its first item in this tile and the
//             wait base = running length offset - tile length prefix at the
//             digit's start.
//   stage     the tile in digit order (its sorted order).
//   phase 2   exclusive length prefix P of the sorted tile (DPP scans within
//             rounds, round and wave totals across); every item writes
//             order and wait = wait base of its digit + P.
// Class totals: a digit holds one class and the sorted tile is class-major,
// so the classes a lane meets over its rounds never decrease. Each lane sums
// its waits in a 128-bit register total and adds it to the class's LDS total
// only when its class changes (and once at the end). Five barriers per tile.

struct FinalFastShared {
  uint64_t stage[T];
  uint16_t cnt[NW][kMaxBins];  // wave counters, then the waves' tile offsets
  uint32_t base_c[kMaxBins];   // output position of the tile's first item of a digit
  uint64_t base_w[kMaxBins];   // wait base of a digit in this tile
  uint64_t wsum[kMaxBins];     // length sums of the tile's digits
  uint64_t clo[256], chi[256]; // class totals, low and high words
  uint32_t part_c[NW + 1];
  uint64_t part_w[NW + 1];
  uint64_t chunk[NW];          // length sum of every wave's share of the sorted tile
};

// Elements of one tile, round-major per wave; items past the end read as zero.
__device__ __forceinline__ void load_final(const uint64_t* keys, int64_t n, int tile,
                                           uint64_t (&e)[K]) {
  const int64_t tb = (int64_t)tile * T;
  const int wb = wave_id() * kWave * K;
  const int lim =
      __builtin_amdgcn_readfirstlane((int)max((int64_t)0, min(n - tb - wb, (int64_t)kWave * K)));
  const __amdgpu_buffer_rsrc_t rk = raw_rsrc(keys + tb + wb, (uint32_t)lim * 8u);
  const int lane = lane_id();
#pragma unroll
  for (int r = 0; r < K; ++r) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rk, (lane + r * kWave) * 8, 0, 0);
    e[r] = ((uint64_t)v[1] << 32) | v[0];
  }
}

template <int NB>  // bits ranked: the final digit has fewer than 2^NB values
__device__ void final_fast(const GArgs& a, int g, FinalFastShared& sh) {
  constexpr int OWN = kMaxBins / NT;  // bins t*OWN .. t*OWN+OWN-1 belong to thread t
  static_assert(OWN == 2, "two bins per thread");
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = t / kWave;
  const int wb = w * kWave * K;
  const Plan* pl = a.plan;
  const int nb = (int)pl->nbins[1];
  const uint32_t d0 = (uint32_t)a.d0;
  const uint32_t psh = pl->wh + d0;
  const uint32_t H = pl->H;
  const uint32_t mh = (1u << pl->wh) - 1;
  const uint32_t lenmask = (1u << psh) - 1;
  const uint32_t hoff = pl->hmin << d0;
  const uint64_t* keys_in = a.keys[0];
  uint16_t* mycnt = sh.cnt[w];
  auto digit = [&](uint32_t key) { return __umul24(key >> psh, H) + ((key >> d0) & mh); };
  auto len = [&](uint32_t key) { return (key & lenmask) + hoff; };

  clear_wave_counters<kMaxBins>(mycnt);
#pragma unroll
  for (int i = 0; i < OWN; ++i) sh.wsum[t * OWN + i] = 0;
  for (int c = t; c < 256; c += NT) sh.clo[c] = sh.chi[c] = 0;
  // running position and wait offsets of the owned digits
  uint32_t carry_c[OWN];
  start_offsets(a, 1, nb, g * kHistRows, carry_c, sh.part_c);
  uint64_t carry_w[OWN];
  {
    uint64_t wv[OWN];
    uint64_t sum = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int b = t * OWN + i;
      wv[i] = b < nb ? a.hist_w[b] : 0ull;
      sum += wv[i];
    }
    uint64_t tot;
    uint64_t ex = block_excl_scan_u64<NT>(sum, sh.part_w, tot);
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int b = t * OWN + i;
      carry_w[i] = ex + (b < nb ? a.block_histw[(size_t)g * kHistRows * kMaxBins + b] : 0ull);
      ex += wv[i];
    }
  }
  // this lane's running wait total and the (relative) class it belongs to
  uint32_t cur = ~0u;
  U128 acc = {0, 0};

  const int tile0 = g * a.fin.tpb;
  const int tile1 = min(a.tiles, tile0 + a.fin.tpb);
  uint64_t e[K];
  load_final(keys_in, a.n, tile0, e);
  for (int tile = tile0; tile < tile1; ++tile) {
    const int64_t tb = (int64_t)tile * T;
    const int cv = (int)min((int64_t)T, a.n - tb);
    const bool full = cv == T;

    // ---- phase 1: digits, tile length sums per digit, ranks -------------
    uint32_t dg[K], rk[K];
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const uint32_t key = (uint32_t)(e[r] >> 32);
      dg[r] = digit(key);
      uint32_t ls = len(key);
      if (!full && wb + r * kWave + lane >= cv) {  // past the end: last digit, no length
        dg[r] = (uint32_t)nb - 1;
        ls = 0;
      }
      atomicAdd((unsigned long long*)&sh.wsum[dg[r]], (unsigned long long)ls);
    }
#pragma unroll
    for (int r = 0; r < K; ++r) rk[r] = rank_round_c<NB>(dg[r], mycnt);
    block_sync();  // counters and length sums are complete; phase 2 of the last tile is over

    // ---- offsets (owners) ---------------------------------------------------
    // The two owned digits are adjacent, so one u32 holds both u16 counters
    // of a wave; counts and offsets stay below 2^16, so packed sums of the
    // pairs never carry from the low half into the high half.
    uint32_t cw[NW];  // wave v's counts of the two owned digits
    uint32_t totp = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      cw[v] = *reinterpret_cast<const u32_alias*>(&sh.cnt[v][t * OWN]);
      totp += cw[v];
    }
    const uint32_t tot[OWN] = {totp & 0xffffu, totp >> 16};
    uint64_t ws[OWN];
    uint32_t local_c = 0;
    uint64_t local_w = 0;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int b = t * OWN + i;
      ws[i] = sh.wsum[b];
      sh.wsum[b] = 0;
      local_c += tot[i];
      local_w += ws[i];
    }
    const uint32_t inc_c = wave_incl_scan_u32(local_c);
    const uint64_t inc_w = wave_incl_scan_u40(local_w);
    if (lane == kWave - 1) {
      sh.part_c[w] = inc_c;
      sh.part_w[w] = inc_w;
    }
    block_sync();
    uint32_t ex_c = inc_c - local_c;
    uint64_t ex_w = inc_w - local_w;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      ex_c += v < w ? sh.part_c[v] : 0u;
      ex_w += v < w ? sh.part_w[v] : 0ull;
    }
    {
      uint32_t run = ex_c | ((ex_c + tot[0]) << 16);
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        *reinterpret_cast<u32_alias*>(&sh.cnt[v][t * OWN]) = run;
        run += cw[v];
      }
    }
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int b = t * OWN + i;
      const uint64_t bw = carry_w[i] - ex_w;
      sh.base_c[b] = carry_c[i] - ex_c;
      sh.base_w[b] = bw;
      carry_c[i] += tot[i];
      carry_w[i] += ws[i];
      ex_c += tot[i];
      ex_w += ws[i];
    }
    block_sync();  // tile offsets and bases are written

    // ---- stage in digit order; load the next tile -------------------------
#pragma unroll
    for (int r = 0; r < K; ++r) rk[r] += mycnt[opaque(dg[r])];
    clear_wave_counters<kMaxBins>(mycnt);
#pragma unroll
    for (int r = 0; r < K; ++r) sh.stage[rk[r]] = e[r];
    if (tile + 1 < tile1) load_final(keys_in, a.n, tile + 1, e);
    block_sync();  // the tile is staged

    // ---- phase 2: tile length prefix, order, waits ---------------------------
    uint32_t lsr[K], inc[K], rt[K];
    uint64_t chunk = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      uint32_t ls = 0;
      if (full || j < cv) ls = len((uint32_t)(sh.stage[j] >> 32));
      lsr[r] = ls;
      inc[r] = wave_incl_scan_u32(ls);  // below 2^32: 64 lengths < 2^26
      rt[r] = (uint32_t)__builtin_amdgcn_readlane((int)inc[r], kWave - 1);
      chunk += rt[r];
    }
    if (lane == 0) sh.chunk[w] = chunk;
    block_sync();
    uint64_t run = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) run += v < w ? sh.chunk[v] : 0ull;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wb + r * kWave + lane;
      if (full || j < cv) {
        const uint64_t x = sh.stage[j];
        const uint32_t key = (uint32_t)(x >> 32);
        const uint32_t c = key >> psh;  // class - pmin
        const uint32_t d = __umul24(c, H) + ((key >> d0) & mh);
        const uint64_t wt = sh.base_w[d] + run + (inc[r] - lsr[r]);
        const uint32_t pos = sh.base_c[d] + (uint32_t)j;
        if (pos < (uint64_t)a.n) {  // always true for consistent counts
          a.order[pos] = (int32_t)(uint32_t)x;
          a.wait[pos] = (int64_t)wt;
        }
        if (c != cur) {
          if (acc.lo | acc.hi) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
          cur = c;
          acc = {0, 0};
        }
        add128(acc, wt);
      }
      run += rt[r];
    }
  }
  if (acc.lo | acc.hi) atomic_add128(sh.clo + cur, sh.chi + cur, acc);

  block_sync();  // every lane's total is in
  uint64_t* clo = sh.clo;
  uint64_t* chi = sh.chi;
  const int P = (int)pl->P;
  for (int c = t; c < P; c += NT) {
    U128 v = {clo[c], chi[c]};
    const int cls = c + (int)pl->pmin;
    if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + cls), a.totals + 2 * (1 + cls) + 1, v);
  }
  if (t == 0) {
    U128 gsum = {0, 0};
    for (int c = 0; c < P; ++c) {
      U128 v = {clo[c], chi[c]};
      add128(gsum, v);
    }
    if (gsum.lo | gsum.hi) atomic_add128(a.totals, a.totals + 1, gsum);
  }
}

// ---- big-tile final pass -----------------------------------------------------
// The fast final pass again, for final digits of at most 256 values (the
// n = 2^26 workload has 160): tiles of 16384 items handled by 1024 threads
// (16 waves x 16 rounds), one workgroup per CU. Four times the items per tile
// means four times longer runs per digit in the scattered writes of order and
// wait, which is what their cost depends on. The thread t < digits owns
// digit t.

constexpr int NTB = 1024;
constexpr int NWB = NTB / kWave;
constexpr int KB = 16;
constexpr int TB = NTB * KB;
constexpr int MAXB = 256;
static_assert(TB == T * kFirstTiles, "blocks of the final split are whole big tiles");

struct FinalBigShared {
  uint64_t stage[TB];
  uint16_t cnt[NWB][MAXB];     // wave counters, then the waves' tile offsets
  uint32_t base_c[MAXB];       // output position of the tile's first item of a digit
  uint64_t base_w[MAXB];       // wait base of a digit in this tile
  uint64_t wsum[MAXB];         // length sums of the tile's digits
  uint64_t clo[256], chi[256]; // class totals, low and high words
  uint32_t part_c[NWB + 1];
  uint64_t part_w[NWB + 1];
  uint64_t chunk[NWB];
};


// Elements of one big tile of `cnt` items at item tb, round-major per wave.
__device__ __forceinline__ void load_final_big(const uint64_t* keys, int64_t tb, int cnt,
                                               uint64_t (&e)[KB]) {
  const int wb = wave_id() * kWave * KB;
  const int lim = __builtin_amdgcn_readfirstlane(max(0, min(cnt - wb, kWave * KB)));
  const __amdgpu_buffer_rsrc_t rk = raw_rsrc(keys + tb + wb, (uint32_t)lim * 8u);
  const int lane = lane_id();
#pragma unroll
  for (int r = 0; r < KB; ++r) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rk, (lane + r * kWave) * 8, 0, 0);
    e[r] = ((uint64_t)v[1] << 32) | v[0];
  }
}

// WIDE: after middle passes (the final digit is u2 >> shift of the last
// pass) or with lengths of 2^26 and more (64 lengths may pass 2^32: the
// round scans are 64-bit and taken again in the store loop instead of being
// held in registers).
template <bool WIDE>
__device__ void final_big(const GArgs& a, int g, FinalBigShared& sh) {
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = wave_id();
  const int wb = w * kWave * KB;
  const Plan* pl = a.plan;
  const int s_last = WIDE ? (int)pl->nscatter - 1 : 1;  // the final pass
  const int nb = (int)pl->nbins[s_last];
  const bool owner = t < nb;
  const uint32_t d0 = (uint32_t)a.d0;
  const uint32_t psh = pl->wh + d0;
  const uint32_t H = pl->H;
  const uint32_t mh = (1u << pl->wh) - 1;
  const uint32_t lenmask = (1u << psh) - 1;
  const uint32_t hoff = pl->hmin << d0;
  const uint32_t sf = WIDE ? pl->shift[s_last] : 0u;
  const uint64_t* keys_in = a.keys[(s_last - 1) & 1];
  uint16_t* mycnt = sh.cnt[w];
  auto digit = [&](uint32_t key) {
    return (__umul24(key >> psh, H) + ((key >> d0) & mh)) >> sf;
  };
  auto len = [&](uint32_t key) { return (key & lenmask) + hoff; };

  clear_wave_counters<MAXB>(mycnt);
  if (t < MAXB) sh.wsum[t] = 0;
  if (t < 256) sh.clo[t] = sh.chi[t] = 0;
  // running position and wait offsets of the owned digit: its global base
  // (exclusive scan of the digit totals) plus the blocks before this one
  uint32_t carry_c;
  uint64_t carry_w;
  {
    const uint32_t c = owner ? a.hist_cnt[s_last * kMaxBins + t] : 0u;
    const uint64_t wv = owner ? a.hist_w[t] : 0ull;
    uint32_t tc;
    uint64_t tw;
    carry_c = block_excl_scan_u32<NTB>(c, sh.part_c, tc);
    carry_w = block_excl_scan_u64<NTB>(wv, sh.part_w, tw);
    if (owner) {
      carry_c += a.block_hist[(size_t)g * kHistRows * kMaxBins + t];
      carry_w += a.block_histw[(size_t)g * kHistRows * kMaxBins + t];
    }
  }
  uint32_t cur = ~0u;  // this lane's running wait total and its class - pmin
  U128 acc = {0, 0};

  const int64_t lo = (int64_t)g * a.fin.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)a.fin.tpb * T);
  uint64_t e[KB];
  load_final_big(keys_in, lo, (int)min((int64_t)TB, hi - lo), e);
  for (int64_t tb = lo; tb < hi; tb += TB) {
    const int cv = (int)min((int64_t)TB, hi - tb);
    const bool full = cv == TB;

    // ---- phase 1: digits, tile length sums per digit, ranks -------------
    // (digits are recomputed where needed: 16 more registers would spill)
    auto digit_of = [&](int r) {
      const uint32_t dd = digit((uint32_t)(opaque((uint32_t)(e[r] >> 32))));
      return (!full && wb + r * kWave + lane >= cv) ? (uint32_t)nb - 1 : dd;  // past the end: last digit
    };
    uint32_t rk[KB];
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const uint32_t key = (uint32_t)(e[r] >> 32);
      const bool past = !full && wb + r * kWave + lane >= cv;
      const uint32_t d = past ? (uint32_t)nb - 1 : digit(key);
      const uint32_t ls = past ? 0u : len(key);
      atomicAdd((unsigned long long*)&sh.wsum[d], (unsigned long long)ls);
      rk[r] = rank_round_c<8>(d, mycnt);
    }
    block_sync();  // counters and length sums are complete; phase 2 of the last tile is over

    // ---- offsets (owners) ---------------------------------------------------
    uint32_t tot = 0;
    uint64_t ws = 0;
    if (owner) {
#pragma unroll
      for (int v = 0; v < NWB; ++v) tot += sh.cnt[v][t];
      ws = sh.wsum[t];
      sh.wsum[t] = 0;
    }
    const uint32_t inc_c = wave_incl_scan_u32(tot);
    // a tile's lengths add up to < 2^40 (lengths below 2^26), else < 2^45
    const uint64_t inc_w = WIDE ? wave_incl_scan_u64(ws) : wave_incl_scan_u40(ws);
    if (lane == kWave - 1) {
      sh.part_c[w] = inc_c;
      sh.part_w[w] = inc_w;
    }
    block_sync();
    uint32_t ex_c = inc_c - tot;
    uint64_t ex_w = inc_w - ws;
#pragma unroll
    for (int v = 0; v < NWB; ++v) {
      ex_c += v < w ? sh.part_c[v] : 0u;
      ex_w += v < w ? sh.part_w[v] : 0ull;
    }
    if (owner) {
      uint32_t run = ex_c;  // counts read again rather than held in 16 registers
#pragma unroll
      for (int v = 0; v < NWB; ++v) {
        const uint32_t c = sh.cnt[v][t];
        sh.cnt[v][t] = (uint16_t)run;
        run += c;
      }
      sh.base_c[t] = carry_c - ex_c;
      sh.base_w[t] = carry_w - ex_w;
      carry_c += tot;
      carry_w += ws;
    }
    block_sync();  // tile offsets and bases are written

    // ---- stage in digit order; load the next tile -------------------------
#pragma unroll
    for (int r = 0; r < KB; ++r) rk[r] += mycnt[digit_of(r)];
    clear_wave_counters<MAXB>(mycnt);
#pragma unroll
    for (int r = 0; r < KB; ++r) sh.stage[rk[r]] = e[r];
    if (tb + TB < hi) load_final_big(keys_in, tb + TB, (int)min((int64_t)TB, hi - tb - TB), e);
    block_sync();  // the tile is staged

    // ---- phase 2: tile length prefix, order, waits, class totals -----------
    auto place = [&](int j, uint64_t wt_in_tile) {
      const uint64_t x = sh.stage[j];
      const uint32_t key = (uint32_t)(x >> 32);
      const uint32_t c = key >> psh;  // class - pmin
      const uint32_t d = digit(key);
      const uint64_t wt = sh.base_w[d] + wt_in_tile;
      const uint32_t pos = sh.base_c[d] + (uint32_t)j;
      if (pos < (uint64_t)a.n) {  // always true for consistent counts
        a.order[pos] = (int32_t)(uint32_t)x;
        a.wait[pos] = (int64_t)wt;
      }
      if (c != cur) {
        if (acc.lo | acc.hi) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
        cur = c;
        acc = {0, 0};
      }
      add128(acc, wt);
    };
    if constexpr (WIDE) {
      uint64_t rt[KB];  // round totals (the scans are taken again below)
      uint64_t chunk = 0;
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        const int j = wb + r * kWave + lane;
        const uint32_t ls = (full || j < cv) ? len((uint32_t)(sh.stage[j] >> 32)) : 0u;
        rt[r] = last_lane_u64(wave_incl_scan_len(ls));
        chunk += rt[r];
      }
      if (lane == 0) sh.chunk[w] = chunk;
      block_sync();
      uint64_t run = 0;
#pragma unroll
      for (int v = 0; v < NWB; ++v) run += v < w ? sh.chunk[v] : 0ull;
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        const int j = wb + r * kWave + lane;
        const bool in_tile = full || j < cv;
        const uint32_t ls = in_tile ? len((uint32_t)(sh.stage[j] >> 32)) : 0u;
        const uint64_t inc = wave_incl_scan_len(ls);
        if (in_tile) place(j, run + (inc - ls));
        run += rt[r];
      }
    } else {
    uint32_t lsr[KB], inc[KB], rt[KB];
    uint64_t chunk = 0;
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const int j = wb + r * kWave + lane;
      uint32_t ls = 0;
      if (full || j < cv) ls = len((uint32_t)(sh.stage[j] >> 32));
      lsr[r] = ls;
      inc[r] = wave_incl_scan_u32(ls);  // below 2^32: 64 lengths < 2^26
      rt[r] = (uint32_t)__builtin_amdgcn_readlane((int)inc[r], kWave - 1);
      chunk += rt[r];
    }
    if (lane == 0) sh.chunk[w] = chunk;
    block_sync();
    uint64_t run = 0;
#pragma unroll
    for (int v = 0; v < NWB; ++v) run += v < w ? sh.chunk[v] : 0ull;
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const int j = wb + r * kWave + lane;
      if (full || j < cv) {
        const uint64_t x = sh.stage[j];
        const uint32_t key = (uint32_t)(x >> 32);
        const uint32_t c = key >> psh;  // class - pmin
        const uint32_t d = __umul24(c, H) + ((key >> d0) & mh);
        const uint64_t wt = sh.base_w[d] + run + (inc[r] - lsr[r]);
        const uint32_t pos = sh.base_c[d] + (uint32_t)j;
        if (pos < (uint64_t)a.n) {  // always true for consistent counts
          a.order[pos] = (int32_t)(uint32_t)x;
          a.wait[pos] = (int64_t)wt;
        }
        if (c != cur) {
          if (acc.lo | acc.hi) atomic_add128(sh.clo + cur, sh.chi + cur, acc);
          cur = c;
          acc = {0, 0};
        }
        add128(acc, wt);
      }
      run += rt[r];
    }
    }
  }
  if (acc.lo | acc.hi) atomic_add128(sh.clo + cur, sh.chi + cur, acc);

  block_sync();  // every lane's total is in
  const int P = (int)pl->P;
  for (int c = t; c < P; c += NTB) {
    U128 v = {sh.clo[c], sh.chi[c]};
    const int cls = c + (int)pl->pmin;
    if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + cls), a.totals + 2 * (1 + cls) + 1, v);
  }
  if (t == 0) {
    U128 gsum = {0, 0};
    for (int c = 0; c < P; ++c) {
      U128 v = {sh.clo[c], sh.chi[c]};
      add128(gsum, v);
    }
    if (gsum.lo | gsum.hi) atomic_add128(a.totals, a.totals + 1, gsum);
  }
}

// ---- compact final pass ------------------------------------------------------
// The big-tile final pass over compact u32 elements. An element holds its
// final digit u2 and the low kChunkBits bits of its id; its first digit d and
// id chunk k come from its position: the first pass left bucket d in id
// order, so bucket d splits into sub-buckets (d, k) of consecutive positions,
// and sub-bucket (d, k) starts at bstart[d] + sub_start[d][k]. These starts
// increase with (d, k); the sub-bucket of a position is the last one whose
// start is not above it (empty sub-buckets share the next one's start, so
// the one found always holds the position). A workgroup copies the starts of
// the buckets its positions span into LDS (`win`) when they fit, narrows them
// per tile, and binary-searches each element's position among them; when
// they do not fit it searches the table in global memory instead.
// Per element: length = ((h + hmin) << d0) + d and id = k << kChunkBits | low
// bits; the staged value carries (u2, d) and the id, the rest is the
// big-tile final pass.

struct FinalCompactShared {
  uint64_t stage[TB];
  uint16_t cnt[NWB][MAXB];     // wave counters, then the waves' tile offsets
  uint32_t base_c[MAXB];       // output position of the tile's first item of a digit
  uint64_t base_w[MAXB];       // wait base of a digit in this tile
  uint64_t flen[MAXB];         // one-bucket tiles: base_c | the digit's length << 32
  uint64_t wsum[MAXB];         // length sums of the tile's digits
  uint64_t clo[256], chi[256]; // class totals, low and high words
  uint32_t bstart[kMaxBins + 1];
  uint32_t win[kWinCap];       // absolute sub-bucket starts of this block's buckets
  uint32_t lbase[MAXB];        // length of a digit's requests without the first digit
  int32_t wd[NWB];             // a wave's one first digit in the tile, or -1
  uint32_t part_c[NWB + 1];
  uint64_t part_w[NWB + 1];
  uint64_t chunk[NWB];
};

__device__ __forceinline__ void load_final_compact(const uint32_t* keys, int64_t tb, int cnt,
                                                   uint32_t (&e)[KB]) {
  const int wb = wave_id() * kWave * KB;
  const int lim = __builtin_amdgcn_readfirstlane(max(0, min(cnt - wb, kWave * KB)));
  const __amdgpu_buffer_rsrc_t rk = raw_rsrc(keys + tb + wb, (uint32_t)lim * 4u);
  const int lane = lane_id();
#pragma unroll
  for (int r = 0; r < KB; ++r)
    e[r] = __builtin_amdgcn_raw_buffer_load_b32(rk, (lane + r * kWave) * 4, 0, 0);
}

// WIN_LDS: the block's sub-bucket starts fit the LDS window and n is below
// kBufferStoreItems; else the starts are read from global memory and the
// outputs stored through plain pointers (separate kernels, see g_final_cglb).
// PAY: the elements carry the caller's ranks (Plan::pay); the totals are
// split by those instead of by the ordering classes.
template <bool WIN_LDS, bool PAY>
__device__ void final_compact(const GArgs& a, int g, FinalCompactShared& sh) {
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int w = wave_id();
  const int wb = w * kWave * KB;
  const Plan* pl = a.plan;
  const int nb = (int)pl->nbins[1];
  const bool owner = t < nb;
  const uint32_t d0 = (uint32_t)a.d0;
  const int nd = 1 << a.d0;
  const uint32_t H = pl->H;
  const uint32_t hmin = pl->hmin;
  const uint32_t magic = div_magic(H);
  const int kpb = a.kpb;
  const uint32_t pay_shift = pl->pay_shift;
  const uint32_t dbits = pay_shift - kChunkBits;  // digit bits (carried ranks above)
  const uint32_t* keys_in = reinterpret_cast<const uint32_t*>(a.keys[0]);
  uint16_t* mycnt = sh.cnt[w];
  auto len_of = [&](uint32_t u2, uint32_t d) {
    return ((u2 - __umul24(class_of(u2, magic), H) + hmin) << d0) + d;
  };

  clear_wave_counters<MAXB>(mycnt);
  if (t < MAXB) {
    sh.wsum[t] = 0;
    sh.lbase[t] = t < nb ? len_of((uint32_t)t, 0u) : 0u;
  }
  if (t < 256) sh.clo[t] = sh.chi[t] = 0;
  bucket_starts<NTB>(a, sh.bstart, sh.part_c);
  uint32_t carry_c;
  uint64_t carry_w;
  {
    const uint32_t c = owner ? a.hist_cnt[kMaxBins + t] : 0u;
    const uint64_t wv = owner ? a.hist_w[t] : 0ull;
    uint32_t tc;
    uint64_t tw;
    carry_c = block_excl_scan_u32<NTB>(c, sh.part_c, tc);
    carry_w = block_excl_scan_u64<NTB>(wv, sh.part_w, tw);
    if (owner) {
      carry_c += a.block_hist[(size_t)g * kHistRows * kMaxBins + t];
      carry_w += a.block_histw[(size_t)g * kHistRows * kMaxBins + t];
    }
  }
  // This lane's running wait total of its current class within the tile
  // (class - pmin = cur; that class's digits end below cur_end). The sorted
  // tile is class-major, so within a tile the classes a lane meets never
  // decrease; the sum goes to the class's LDS total at every class change
  // and at the end of the tile. A lane's 16 waits of a tile stay below 2^61,
  // so the sum fits 64 bits.
  uint32_t cur = ~0u, cur_end = 0;
  uint64_t acc64 = 0;
  auto flush_class = [&]() {
    if (acc64) atomic_add128(sh.clo + cur, sh.chi + cur, U128{acc64, 0});
    acc64 = 0;
  };

  const int64_t lo = (int64_t)g * a.fin.tpb * T;
  const int64_t hi = min(a.n, lo + (int64_t)a.fin.tpb * T);
  // sub-bucket starts of the buckets [d_lo, d_hi] that this block's positions span
  const int d_lo = hi > lo ? bucket_of(sh.bstart, nd, (uint32_t)lo) : 0;
  const int d_hi = hi > lo ? bucket_of(sh.bstart, nd, (uint32_t)(hi - 1)) : 0;
  const int win0 = d_lo << kpb;
  const int wn = (d_hi - d_lo + 1) << kpb;
  if (WIN_LDS != (wn <= kWinCap && a.n < kBufferStoreItems)) return;  // the other kernel's block
  if (WIN_LDS) {
    for (int j = t; j < wn; j += NTB)
      sh.win[j] = sh.bstart[(win0 + j) >> kpb] + a.sub_start[win0 + j];
  }
  block_sync();
  auto sb = [&](int j) -> uint32_t {
    return WIN_LDS ? sh.win[j] : sh.bstart[(win0 + j) >> kpb] + a.sub_start[win0 + j];
  };
  // last j in [jl, jh] with sb(j) <= pos, given sb(jl) <= pos: binary
  // lifting with steps from the largest power of two <= jh - jl down to 1
  // (jl and jh are uniform, so the trip count is)
  auto find = [&](uint32_t pos, int jl, int jh) {
    const int span = jh - jl;
    for (int step = span > 0 ? 1 << (31 - __clz(span)) : 0; step > 0; step >>= 1) {
      const int c = min(jl + step, jh);
      if (sb(c) <= pos) jl = c;
    }
    return jl;
  };

  // The elements of tile t + 1 are loaded before the stores of tile t, and
  // ranked (at the top of the next iteration) after them. The compiler then
  // sees the loads, the (exactly counted, unconditional) stores and the first
  // use of the loads in that order, and waits only for the loads: the stores
  // drain while the next tile is ranked.
  uint32_t e[KB];   // elements of the tile being ranked
  // per item: rank (below 2^14) | window index << 14 (below 2^18; with the
  // LDS window below 2^9, and then the final digit follows at bit 23)
  uint32_t rw[KB];
  static_assert(kWinCap <= 512, "window index, rank and digit share 32 bits");
  // output resources (used when n < kBufferStoreItems: byte offsets below 2^31)
  const __amdgpu_buffer_rsrc_t rs_order = raw_rsrc(a.order, (uint32_t)a.n * 4u);
  const __amdgpu_buffer_rsrc_t rs_wait = raw_rsrc(a.wait, (uint32_t)a.n * 8u);
  auto tile_items = [&](int64_t tb) { return (int)min((int64_t)TB, hi - tb); };
  auto digit_of = [&](int r, int cv) {  // past the end: the last digit
    return (cv < TB && wb + r * kWave + lane >= cv) ? (uint32_t)nb - 1
                                                   : __builtin_amdgcn_ubfe(e[r], kChunkBits, dbits);
  };
  // ---- phase 1: decode, tile length sums per digit, ranks --------------
  // (Ballot matching here: with at most 256 final digits many lanes of a
  // round share a digit, and the lane-mask ranking of the first pass then
  // serialises on its LDS atomics.)
  // A wave whose full share of the tile lies in one first-digit bucket d
  // (nearly all: a bucket spans about n / 2^d0 positions) adds no lengths
  // here: its requests of digit u2 contribute count * (lbase[u2] + d), which
  // the digit's owner forms from the wave's counter. The other waves add each
  // length to the digit's LDS sum.
  // Full tiles whose positions all lie in one first-digit bucket d (nearly
  // all: a bucket spans about n / 2^d0 positions) hold one length per final
  // digit u2, lbase[u2] + d. The k-th request of u2 in such a tile then waits
  // (wait of u2's first request in the tile) + k * length, so no length scan
  // is needed, and the owner of u2 adds the digit's share of its class total
  // in closed form: count * first wait + length * count * (count - 1) / 2.
  bool tile_one = false;
  U128 own_tot = {0, 0};  // owners: closed-form class-total shares of their digit
  auto phase1 = [&](int64_t tb) {
    const int cv = tile_items(tb);
    // the sub-buckets this tile's positions lie in, then those of this wave's
    // share (usually one: a wave covers 1024 positions); the bounds are
    // uniform, so the searches below have uniform trip counts
    const int ja = __builtin_amdgcn_readfirstlane(find((uint32_t)tb, 0, wn - 1));
    const int jb = __builtin_amdgcn_readfirstlane(find((uint32_t)(tb + cv - 1), ja, wn - 1));
    tile_one = !PAY && cv == TB && ((win0 + ja) >> kpb) == ((win0 + jb) >> kpb);
    const uint32_t wlast = (uint32_t)(tb + cv - 1);
    const int wja = __builtin_amdgcn_readfirstlane(
        find(min((uint32_t)(tb + wb), wlast), ja, jb));
    const int wjb = __builtin_amdgcn_readfirstlane(
        find(min((uint32_t)(tb + wb + kWave * KB - 1), wlast), wja, jb));
    const int wda = (win0 + wja) >> kpb;
    const bool one_digit = wda == ((win0 + wjb) >> kpb) && wb + kWave * KB <= cv;  // uniform
    if (lane == 0) sh.wd[w] = one_digit ? wda : -1;
    auto rank_items = [&](auto add_lengths) {
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        const int j = wb + r * kWave + lane;
        const uint32_t jj = (uint32_t)find((uint32_t)(tb + j), wja, wjb);
        const uint32_t dg = digit_of(r, cv);
        if constexpr (decltype(add_lengths)::value) {
          const uint32_t d = (uint32_t)((win0 + (int)jj) >> kpb);
          const uint32_t ls = j >= cv ? 0u : sh.lbase[dg] + d;
          atomicAdd((unsigned long long*)&sh.wsum[dg], (unsigned long long)ls);
        }
        rw[r] = rank_round_c<8>(dg, mycnt) | (jj << 14) | (WIN_LDS ? dg << 23 : 0u);
      }
    };
    if (one_digit)
      rank_items(std::false_type{});
    else
      rank_items(std::true_type{});
  };

  load_final_compact(keys_in, lo, tile_items(lo), e);
  for (int64_t tb = lo; tb < hi; tb += TB) {
    phase1(tb);
    const int cv = tile_items(tb);
    const bool full = cv == TB;
    block_sync();  // counters and length sums are complete; phase 2 of the last tile is over

    // ---- offsets (owners) ---------------------------------------------------
    uint32_t tot = 0;
    uint64_t ws = 0;
    if (owner) {
      const uint32_t lb = sh.lbase[t];
#pragma unroll
      for (int v = 0; v < NWB; ++v) {
        const uint32_t c = sh.cnt[v][t];
        const int dv = sh.wd[v];
        tot += c;
        if (dv >= 0) ws += (uint64_t)c * (lb + (uint32_t)dv);
      }
      ws += sh.wsum[t];
      sh.wsum[t] = 0;
    }
    const uint32_t inc_c = wave_incl_scan_u32(tot);
    const uint64_t inc_w = wave_incl_scan_u40(ws);  // a tile's lengths add up to < 2^40
    if (lane == kWave - 1) {
      sh.part_c[w] = inc_c;
      sh.part_w[w] = inc_w;
    }
    block_sync();
    uint32_t ex_c = inc_c - tot;
    uint64_t ex_w = inc_w - ws;
    for (int v = 0; v < w; ++v) {  // (w is uniform)
      ex_c += sh.part_c[v];
      ex_w += sh.part_w[v];
    }
    const bool one = tile_one;  // (uniform)
    if (owner) {
      uint32_t run = ex_c;
#pragma unroll
      for (int v = 0; v < NWB; ++v) {
        const uint32_t c = sh.cnt[v][t];
        sh.cnt[v][t] = (uint16_t)run;
        run += c;
      }
      sh.base_c[t] = carry_c - ex_c;
      if (one) {
        const uint32_t len = sh.lbase[t] + (uint32_t)sh.wd[0];
        sh.flen[t] = ((uint64_t)len << 32) | (carry_c - ex_c);
        sh.base_w[t] = carry_w - (uint64_t)ex_c * len;
        // the digit's waits in this tile: carry_w + k * len for k < tot
        add128(own_tot, U128{(uint64_t)tot * carry_w, __umul64hi((uint64_t)tot, carry_w)});
        add128(own_tot, (uint64_t)len * ((uint64_t)tot * (tot - 1) / 2));
      } else {
        sh.base_w[t] = carry_w - ex_w;
      }
      carry_c += tot;
      carry_w += ws;
    }
    block_sync();  // tile offsets and bases are written

    // ---- stage (digit, first digit, id) in digit order; load the next tile ---
    uint32_t rk[KB];
#pragma unroll
    for (int r = 0; r < KB; ++r)
      rk[r] = (rw[r] & 0x3fffu) + mycnt[opaque(WIN_LDS ? rw[r] >> 23 : digit_of(r, cv))];
    clear_wave_counters<MAXB>(mycnt);
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const int idx = win0 + (int)((rw[r] >> 14) & (WIN_LDS ? 511u : 0x3ffffu));
      const uint32_t d = (uint32_t)(idx >> kpb);
      const uint32_t id = ((uint32_t)(idx & ((1 << kpb) - 1)) << kChunkBits) |
                          (e[r] & ((1u << kChunkBits) - 1));
      const uint32_t rank_bits = PAY ? (e[r] >> pay_shift) << 18 : 0u;
      const uint32_t dg = WIN_LDS ? rw[r] >> 23 : digit_of(r, cv);
      sh.stage[rk[r]] = ((uint64_t)(rank_bits | (dg << 10) | d) << 32) | id;
    }
    const bool more = tb + TB < hi;
    if (more) load_final_compact(keys_in, tb + TB, tile_items(tb + TB), e);
    block_sync();  // the tile is staged

    if (one) {
      // ---- phase 2, one-bucket tile: waits in closed form ------------------
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        const int j = wb + r * kWave + lane;
        const uint64_t x = sh.stage[j];
        const uint64_t f = sh.flen[(uint32_t)(x >> 42)];
        const uint64_t wt = sh.base_w[(uint32_t)(x >> 42)] + (uint64_t)(uint32_t)j * (f >> 32);
        const uint32_t pos = (uint32_t)f + (uint32_t)j;
        const bool item = pos < (uint64_t)a.n;  // (pos < n for consistent counts)
        if constexpr (WIN_LDS) {
          const uint32_t slot = item ? pos : (uint32_t)a.n;
          __builtin_amdgcn_raw_buffer_store_b32((uint32_t)x, rs_order, slot * 4u, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b64(u32x2{(uint32_t)wt, (uint32_t)(wt >> 32)},
                                                rs_wait, slot * 8u, 0, 0);
        } else {
          int32_t* po = item ? a.order + pos : reinterpret_cast<int32_t*>(a.sink);
          int64_t* pw = item ? a.wait + pos : reinterpret_cast<int64_t*>(a.sink + 1);
          *po = (int32_t)(uint32_t)x;
          *pw = (int64_t)wt;
        }
      }
      continue;
    }
    // ---- phase 2: tile length prefix, order, waits, class totals -----------
    uint32_t exc[KB], rt[KB];  // exclusive length prefix within the round; round total
    uint64_t chunk = 0;
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const int j = wb + r * kWave + lane;
      uint32_t ls = 0;
      if (full || j < cv) {
        const uint32_t hw = (uint32_t)(sh.stage[j] >> 32);
        ls = sh.lbase[PAY ? (hw >> 10) & (MAXB - 1) : hw >> 10] + (hw & 1023u);
      }
      const uint32_t inc = wave_incl_scan_u32(ls);  // below 2^32: 64 lengths < 2^26
      exc[r] = inc - ls;
      rt[r] = (uint32_t)__builtin_amdgcn_readlane((int)inc, kWave - 1);
      chunk += rt[r];
    }
    if (lane == 0) sh.chunk[w] = chunk;
    block_sync();
    uint64_t run = 0;
    for (int v = 0; v < w; ++v) run += sh.chunk[v];  // (w is uniform)
    // Stores are unconditional, so that the compiler counts them exactly:
    // lanes without an item (past the end of the last, partial tile) store
    // at the end of the buffer resource, where the range check drops the
    // store, or write to the sink (plain pointers).
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const int j = wb + r * kWave + lane;
      const uint64_t x = sh.stage[j];
      const uint32_t u2 = PAY ? (uint32_t)(x >> 42) & (MAXB - 1) : (uint32_t)(x >> 42);
      const uint64_t wt = sh.base_w[u2] + run + exc[r];
      const uint32_t pos = sh.base_c[u2] + (uint32_t)j;
      const bool in_tile = full || j < cv;
      const bool item = in_tile && pos < (uint64_t)a.n;  // (pos < n for consistent counts)
      if constexpr (WIN_LDS) {
        const uint32_t slot = item ? pos : (uint32_t)a.n;
        __builtin_amdgcn_raw_buffer_store_b32((uint32_t)x, rs_order, slot * 4u, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{(uint32_t)wt, (uint32_t)(wt >> 32)}, rs_wait,
                                              slot * 8u, 0, 0);
      } else {
        int32_t* po = item ? a.order + pos : reinterpret_cast<int32_t*>(a.sink);
        int64_t* pw = item ? a.wait + pos : reinterpret_cast<int64_t*>(a.sink + 1);
        *po = (int32_t)(uint32_t)x;
        *pw = (int64_t)wt;
      }
      if (in_tile) {
        if constexpr (PAY) {  // the carried rank, in no particular order
          const uint32_t c = (uint32_t)(x >> 50);
          if (c != cur) {
            if (cur != ~0u) flush_class();
            cur = c;
          }
        } else if (u2 >= cur_end) {  // a new class for this lane
          if (cur != ~0u) flush_class();
          cur = class_of(u2, magic);  // class - pmin
          cur_end = __umul24(cur + 1, H);
        }
        acc64 += wt;
      }
      run += rt[r];
    }
    if (cur != ~0u) flush_class();  // the next tile starts again at the first class
    cur = ~0u;
    cur_end = 0;
  }
  if (owner && (own_tot.lo | own_tot.hi)) {
    const uint32_t c = class_of((uint32_t)t, magic);
    atomic_add128(sh.clo + c, sh.chi + c, own_tot);
  }
  block_sync();  // every lane's total is in
  // (carried ranks are the caller's ranks themselves)
  const int P = PAY ? (int)*a.pay_pmax + 1 : (int)pl->P;
  for (int c = t; c < P; c += NTB) {
    U128 v = {sh.clo[c], sh.chi[c]};
    const int cls = c + (PAY ? 0 : (int)pl->pmin);
    if (v.lo | v.hi) atomic_add128(a.totals + 2 * (1 + cls), a.totals + 2 * (1 + cls) + 1, v);
  }
  if (t == 0) {
    U128 gsum = {0, 0};
    for (int c = 0; c < P; ++c) {
      U128 v = {sh.clo[c], sh.chi[c]};
      add128(gsum, v);
    }
    if (gsum.lo | gsum.hi) atomic_add128(a.totals, a.totals + 1, gsum);
  }
}

__global__ __launch_bounds__(NTB) void g_final_big(GArgs a) {
  __shared__ union {
    FinalBigShared big;
    FinalCompactShared compact;
  } sh;
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  if (pl->compact) {
    if (!pl->pay) final_compact<true, false>(a, blockIdx.x, sh.compact);
    return;
  }
  if (!use_big_final(pl)) return;
  final_big<false>(a, blockIdx.x, sh.big);
}

// The compact final pass for the blocks whose sub-bucket starts do not fit
// the LDS window (rare: a block must span hundreds of first-digit buckets);
// they are searched in global memory. A kernel of its own, so that the common
// kind's loop holds no global loads besides the element prefetch and the
// compiler's wait counts stay exact there. Returns at once for other blocks.
__global__ __launch_bounds__(NTB) void g_final_cglb(GArgs a) {
  __shared__ union {
    FinalCompactShared compact;
    FinalBigShared big;
  } sh;
  const Plan* pl = a.plan;
  if (!pl->ok) return;
  if (use_wide_big_final(a, pl)) {
    final_big<true>(a, blockIdx.x, sh.big);
    return;
  }
  if (!pl->compact || pl->pay || !pl->cglb) return;
  final_compact<false, false>(a, blockIdx.x, sh.compact);
}

// The compact final pass with carried ranks, in kernels of their own (one
// kernel holding both forms would spill registers), launched only when the
// caller passed ranks to carry.
__global__ __launch_bounds__(NTB) void g_final_pay(GArgs a) {
  __shared__ FinalCompactShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || !pl->compact || !pl->pay) return;
  final_compact<true, true>(a, blockIdx.x, sh);
}

__global__ __launch_bounds__(NTB) void g_final_pay_cglb(GArgs a) {
  __shared__ FinalCompactShared sh;
  const Plan* pl = a.plan;
  if (!pl->ok || !pl->compact || !pl->pay || !pl->cglb) return;
  final_compact<false, true>(a, blockIdx.x, sh);
}

template <typename unused = void>
__global__ __launch_bounds__(NT, kScatterWavesPerSimd) void g_final(GArgs a) {
  __shared__ union {
    FinalShared generic;
    FinalFastShared fast;
  } sh;
  const Plan* pl = a.plan;
  if (!pl->ok || pl->compact || use_big_final(pl) || use_wide_big_final(a, pl)) return;
  if (pl->packed && pl->W == 32 && pl->nscatter == 2 && pl->small) {
    if (pl->nbits[1] <= 8)
      final_fast<8>(a, blockIdx.x, sh.fast);
    else
      final_fast<10>(a, blockIdx.x, sh.fast);
  } else
    final_generic(a, blockIdx.x, sh.generic);
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

// Blocks of whole tiles, tpb a multiple of `mult` tiles, at most `resident`
// blocks (the workgroups that fit on the device at once).
Split make_split(int64_t n, int resident, int mult) {
  const int64_t tiles = (n + T - 1) / T;
  const int64_t chunks = (tiles + mult - 1) / mult;
  int64_t g = resident;
  if (g > kMaxBlocks) g = kMaxBlocks;
  if (g > chunks) g = chunks;
  if (g < 1) g = 1;
  Split s;
  s.tpb = (int32_t)((chunks + g - 1) / g * mult);
  s.blocks = (int32_t)((tiles + s.tpb - 1) / s.tpb);
  return s;
}

void mark(const StageEvents* ev, int stage, bool after, hipStream_t st) {
  if (!ev) return;
  hipEvent_t e = after ? ev->after[stage] : ev->before[stage];
  if (e) (void)hipEventRecord(e, st);
}

}  // namespace

Split global_first_split(int64_t n) {
  static const int r = resident_blocks(reinterpret_cast<const void*>(g_first<10>), NT);
  return make_split(n, r, kFirstTiles);
}

Split global_final_split(int64_t n) {
  static const int r = resident_blocks(reinterpret_cast<const void*>(g_final_big), NTB);
  return make_split(n, r, kFirstTiles);
}

Split global_mid_split(int64_t n) {
  static const int r = resident_blocks(reinterpret_cast<const void*>(g_mid), NT);
  return make_split(n, r, kFirstTiles);  // the fast middle pass walks big tiles
}

hipError_t launch_global_schedule(const GArgs& a, hipStream_t st, const StageEvents* ev) {
  const int vec_ok = ((uintptr_t)a.priority % 4 == 0) && ((uintptr_t)a.length % 16 == 0);
  const dim3 gm(a.main.blocks);
  const dim3 gmh(a.main.blocks * kHistRows);
  mark(ev, 0, false, st);
  hipLaunchKernelGGL(g_hist0, gmh, dim3(HT), 0, st, a, vec_ok);
  mark(ev, 0, true, st);
  hipLaunchKernelGGL(g_scan, dim3((1u << a.d0) + 1), dim3(SCT), 0, st, a, 0);
  mark(ev, 1, false, st);
  if (a.d0 == 9)
    hipLaunchKernelGGL(g_first<9>, gm, dim3(NT), 0, st, a);
  else if (a.d0 == 10)
    hipLaunchKernelGGL(g_first<10>, gm, dim3(NT), 0, st, a);
  else
    hipLaunchKernelGGL(g_first<8>, gm, dim3(NT), 0, st, a);
  mark(ev, 1, true, st);
  mark(ev, 6, false, st);
  if (a.split_mid) {
    // Ranks below 2^8 and lengths below 2^31 make the mixed-radix value
    // below 2^(39 - d0), so at most (38 - d0) / 10 middle passes of 10 bits.
    const int max_mids = (38 - a.d0) / 10;
    for (int s = 1; s <= max_mids && s < kMaxScatter - 1; ++s) {
      hipLaunchKernelGGL(g_mid_count, dim3(a.mid.blocks), dim3(NT), 0, st, a, s);
      hipLaunchKernelGGL(g_mid_scan, dim3(kMaxBins / 4), dim3(NT), 0, st, a, s);
      hipLaunchKernelGGL(g_mid_scatter, dim3(a.mid.blocks), dim3(NT), 0, st, a, s);
    }
  } else {
    hipLaunchKernelGGL(g_mid, dim3(a.mid.blocks), dim3(NT), 0, st, a);
  }
  mark(ev, 6, true, st);
  const dim3 gf(a.fin.blocks);
  hipLaunchKernelGGL(g_histF, dim3(a.fin.blocks * kHistRows), dim3(HT), 0, st, a);
  hipLaunchKernelGGL(g_scan, dim3(kMaxBins + 1), dim3(SCT), 0, st, a, 1);
  mark(ev, 2, false, st);
  // exactly one of the two does the work; the plan on the device decides
  hipLaunchKernelGGL(g_final_big, gf, dim3(NTB), 0, st, a);
  if (a.chunked) hipLaunchKernelGGL(g_final_cglb, gf, dim3(NTB), 0, st, a);
  if (a.chunked && a.payload) {
    hipLaunchKernelGGL(g_final_pay, gf, dim3(NTB), 0, st, a);
    hipLaunchKernelGGL(g_final_pay_cglb, gf, dim3(NTB), 0, st, a);
  }
  hipLaunchKernelGGL(g_final<>, gf, dim3(NT), 0, st, a);
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
