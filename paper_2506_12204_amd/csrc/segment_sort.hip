// LDS-resident schedule of whole queues, one workgroup per queue.
//
// A queue of m <= NT*K requests is read once from HBM, ordered by
// (priority, length, id) with an LSD radix sort that never leaves LDS, and
// its waits and totals are written once: 5 bytes read and 12 bytes written
// per request, plus the queue's totals. This is the drained min-heap of
// Algorithm 1 (MinHeap Construction) for a whole snapshot of the queue, with
// the waiting times of Eq. 1 as the exclusive prefix of service times.
//
// Layout inside the workgroup: wave w owns positions [w*64*kr, (w+1)*64*kr)
// in kr rounds of 64 consecutive positions (lane = position within the
// round). Every LSD pass ranks digits stably in that position order, so ids
// (the arrival index, kept in the low 16 bits of each element) break ties
// without ever being sorted on.
#include "block_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int kIdBits = 16;  // local ids < SEM_SEGMENT_CAP = 16384 < 2^16

template <int NT, int K, int DMAX>
struct SegShared {
  static constexpr int NW = NT / kWave;
  static constexpr int CAP = NT * K;
  static constexpr int STRIDE = 1 << DMAX;
  static_assert(NW * STRIDE * 2 <= CAP * 8, "counters must fit in the stage");
  uint64_t stage[CAP];  // elements; the wave counters alias its front
  uint32_t excl[STRIDE + 1];
  uint64_t cls_lo[256];
  uint64_t cls_hi[256];
  uint32_t red[4][NW];
  uint64_t scan64[NW + 1];
  uint32_t scan32[NW + 1];
};

// Per-thread run of consecutive schedule positions in one class, added into
// the workgroup's per-class LDS accumulators when the class changes.
__device__ __forceinline__ void flush_run(uint64_t* lo, uint64_t* hi, int cls,
                                          U128& acc) {
  if (cls >= 0 && (acc.lo | acc.hi)) atomic_add128(lo + cls, hi + cls, acc);
  acc.lo = acc.hi = 0;
}

template <int NT, int K, int DMAX>
__global__ __launch_bounds__(NT) void segment_schedule_kernel(SegArgs a) {
  using SH = SegShared<NT, K, DMAX>;
  constexpr int NW = SH::NW;
  constexpr int STRIDE = SH::STRIDE;
  __shared__ SH sh;
  u16_alias* cnt = reinterpret_cast<u16_alias*>(sh.stage);

  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int tot_stride = 1 + a.num_classes;

  if (blockIdx.x == 0 && threadIdx.x == 0 && a.offsets) {
    if (a.offsets[0] != 0 || a.offsets[a.num_segments] != a.n_total)
      atomicOr(a.flags, kFlagInval);
  }

  for (int64_t s = blockIdx.x; s < a.num_segments; s += gridDim.x) {
    const int64_t base = a.offsets ? a.offsets[s] : 0;
    const int64_t m64 = a.offsets ? a.offsets[s + 1] - base : a.n_total;
    if (m64 < 0 || m64 > a.max_segment || base < 0 || base + m64 > a.n_total) {
      if (threadIdx.x == 0) atomicOr(a.flags, kFlagInval);
      continue;
    }
    if (m64 <= a.route_lo || m64 > a.route_hi) continue;
    const int m = (int)m64;
    uint64_t* tot = a.totals + 2 * (s * tot_stride);

    if (m == 0) {
      for (int c = threadIdx.x; c < 2 * tot_stride; c += NT) tot[c] = 0;
      continue;
    }

    const int kr = (m + NT - 1) / NT;  // rounds per wave, <= K
    const int wbase = w * kWave * kr;

    // ---- load (coalesced per round) and range checks -------------------
    // el[r] first holds the raw request (priority << 32 | length), then its key.
    uint64_t el[K];
    uint32_t lmin = 0xffffffffu, lmax = 0, pmin = 0xffu, pmax = 0, bad = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      el[r] = 0;
      if (r < kr) {
        const int i = wbase + r * kWave + lane;
        if (i < m) {
          const uint32_t p = a.priority[base + i];
          const int32_t l = a.length[base + i];
          if (l < 0 || (int)p >= a.num_classes) bad = 1;
          lmin = min(lmin, (uint32_t)l);
          lmax = max(lmax, (uint32_t)l);
          pmin = min(pmin, p);
          pmax = max(pmax, p);
          el[r] = ((uint64_t)p << 32) | (uint32_t)l;
        }
      }
    }
    lmin = wave_min_u32(lmin);
    lmax = wave_max_u32(lmax);
    pmin = wave_min_u32(pmin);
    pmax = wave_max_u32(pmax);
    bad = wave_or_u32(bad);
    block_sync();  // previous segment's use of `red` is over
    if (lane == 0) {
      sh.red[0][w] = lmin;
      sh.red[1][w] = lmax;
      sh.red[2][w] = pmin;
      sh.red[3][w] = pmax | (bad << 31);
    }
    for (int c = threadIdx.x; c < 256; c += NT) sh.cls_lo[c] = sh.cls_hi[c] = 0;
    block_sync();
    lmin = 0xffffffffu;
    lmax = 0;
    pmin = 0xffu;
    pmax = 0;
    bad = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      lmin = min(lmin, sh.red[0][i]);
      lmax = max(lmax, sh.red[1][i]);
      pmin = min(pmin, sh.red[2][i]);
      pmax = max(pmax, sh.red[3][i] & 0xffu);
      bad |= sh.red[3][i] >> 31;
    }
    if (bad) {
      if (threadIdx.x == 0) atomicOr(a.flags, kFlagRange);
      continue;
    }

    // ---- key: (priority - pmin, length - lmin) as two bit fields ----------
    const uint32_t wl = bit_width32(lmax - lmin);
    const uint32_t wp = bit_width32(pmax - pmin);
    const uint32_t kb = wl + wp;
    const uint64_t kmax = kb ? ((1ull << kb) - 1) : 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int i = wbase + r * kWave + lane;
      const uint32_t p = (uint32_t)(el[r] >> 32);
      const uint32_t l = (uint32_t)el[r];
      const uint64_t key = (r < kr && i < m) ? ((uint64_t)(p - pmin) << wl) | (l - lmin)
                                             : kmax;  // padding sorts last (it sits last)
      el[r] = (key << kIdBits) | (uint32_t)(i & 0xffff);
    }

    // ---- LSD radix passes in LDS ------------------------------------------
    const int npass = kb ? (int)((kb + DMAX - 1) / DMAX) : 0;
    const int dstep = npass ? (int)((kb + npass - 1) / npass) : 0;
    for (int q = 0; q < npass; ++q) {
      const int shift = q * dstep;
      const int nb = min(dstep, (int)kb - shift);
      const int nbins = 1 << nb;
      block_sync();  // the stage (aliased by the counters) is free
      for (int b = lane; b < nbins; b += kWave) cnt[w * STRIDE + b] = 0;
      // a wave only touches its own counter row until the next barrier
      uint32_t dg[K], rk[K];
#pragma unroll
      for (int r = 0; r < K; ++r) {
        if (r < kr) {
          dg[r] = (uint32_t)(el[r] >> (kIdBits + shift)) & (uint32_t)(nbins - 1);
          rk[r] = rank_round(dg[r], nb, cnt + w * STRIDE);
        }
      }
      block_sync();
      block_digit_offsets<NT>(cnt, STRIDE, nbins, sh.excl, sh.scan32);
#pragma unroll
      for (int r = 0; r < K; ++r)
        if (r < kr) rk[r] += sh.excl[dg[r]] + cnt[w * STRIDE + dg[r]];
      block_sync();  // every counter read happens before the stage writes
#pragma unroll
      for (int r = 0; r < K; ++r)
        if (r < kr) sh.stage[rk[r]] = el[r];
      block_sync();
#pragma unroll
      for (int r = 0; r < K; ++r)
        if (r < kr) el[r] = sh.stage[wbase + r * kWave + lane];
    }

    // ---- waits: exclusive scan of lengths in schedule order ---------------
    const uint64_t lmask = wl ? ((1ull << wl) - 1) : 0;
    uint64_t len_s[K];
    uint64_t wsum = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const int j = wbase + r * kWave + lane;
      len_s[r] = 0;
      if (r < kr && j < m) len_s[r] = ((el[r] >> kIdBits) & lmask) + lmin;
      wsum += len_s[r];
    }
    // wave totals -> exclusive offsets of the waves
    uint64_t wtot = wave_incl_scan_u64(wsum);
    wtot = last_lane_u64(wtot);
    uint64_t dummy;
    uint64_t run = block_excl_scan_u64<NT>(lane == 0 ? wtot : 0, sh.scan64, dummy);
    run = __shfl(run, 0, kWave);

    int cur = -1;
    U128 acc = {0, 0};
#pragma unroll
    for (int r = 0; r < K; ++r) {
      if (r < kr) {
        const int j = wbase + r * kWave + lane;
        const uint64_t incl = wave_incl_scan_len((uint32_t)len_s[r]);
        const uint64_t wt = run + incl - len_s[r];
        run += last_lane_u64(incl);
        if (j < m) {
          const uint64_t key = el[r] >> kIdBits;
          const int cls = (int)((key >> wl) + pmin);
          a.order[base + j] = (int32_t)(el[r] & 0xffff);
          a.wait[base + j] = (int64_t)wt;
          if (cls != cur) {
            flush_run(sh.cls_lo, sh.cls_hi, cur, acc);
            cur = cls;
          }
          add128(acc, wt);
        }
      }
    }
    flush_run(sh.cls_lo, sh.cls_hi, cur, acc);
    block_sync();

    // ---- totals of this queue ------------------------------------------------
    for (int c = threadIdx.x; c < a.num_classes; c += NT) {
      tot[2 * (1 + c)] = sh.cls_lo[c];
      tot[2 * (1 + c) + 1] = sh.cls_hi[c];
    }
    if (threadIdx.x == 0) {
      U128 g = {0, 0};
      for (uint32_t c = pmin; c <= pmax; ++c) {
        U128 v = {sh.cls_lo[c], sh.cls_hi[c]};
        add128(g, v);
      }
      tot[0] = g.lo;
      tot[1] = g.hi;
    }
  }
}

}  // namespace

template <int NT, int K, int DMAX>
static hipError_t launch_one(const SegArgs& a, int grid, hipStream_t st) {
  hipLaunchKernelGGL((segment_schedule_kernel<NT, K, DMAX>), dim3(grid), dim3(NT), 0,
                     st, a);
  return hipGetLastError();
}

hipError_t launch_segment_schedule(SegArgs a, SegSize size, int grid, hipStream_t st) {
  switch (size) {
    case SegSize::kTiny:
      a.route_lo = -1;
      a.route_hi = kSegTinyCap;
      return launch_one<64, 4, 8>(a, grid, st);
    case SegSize::kSmall:
      a.route_lo = kSegTinyCap;
      a.route_hi = kSegSmallCap;
      return launch_one<256, 4, 8>(a, grid, st);
    case SegSize::kMedium:
      a.route_lo = kSegSmallCap;
      a.route_hi = kSegMediumCap;
      return launch_one<256, 16, 8>(a, grid, st);
    case SegSize::kLarge:
    default:
      a.route_lo = kSegMediumCap;
      a.route_hi = kSegLargeCap;
      return launch_one<512, 32, 10>(a, grid, st);
  }
}

}  // namespace semsched
