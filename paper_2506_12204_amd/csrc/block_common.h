// Workgroup-level building blocks for the gfx950 scheduling kernels: block
// scans and the conversion of per-wave digit counters into stable in-block
// digit offsets. Every function here contains __syncthreads() and must be
// reached by all threads of the workgroup.
#pragma once

#include "device_common.h"

namespace semsched {

// Exclusive scan of one u32 per thread across the workgroup (thread order).
// `scratch` holds at least NT/64 + 1 u32 of LDS. Returns the exclusive prefix;
// `total` receives the sum over the workgroup.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan_u32(uint32_t v, uint32_t* scratch,
                                                        uint32_t& total) {
  constexpr int NW = NT / kWave;
  const int w = threadIdx.x / kWave;
  const uint32_t incl = wave_incl_scan_u32(v);
  if (lane_id() == kWave - 1) scratch[w] = incl;
  block_sync();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t s = scratch[i];
    off += (i < w) ? s : 0u;
    tot += s;
  }
  block_sync();
  total = tot;
  return off + incl - v;
}

template <int NT>
__device__ __forceinline__ uint64_t block_excl_scan_u64(uint64_t v, uint64_t* scratch,
                                                        uint64_t& total) {
  constexpr int NW = NT / kWave;
  const int w = threadIdx.x / kWave;
  const uint64_t incl = wave_incl_scan_u64(v);
  if (lane_id() == kWave - 1) scratch[w] = incl;
  block_sync();
  uint64_t off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint64_t s = scratch[i];
    off += (i < w) ? s : 0u;
    tot += s;
  }
  block_sync();
  total = tot;
  return off + incl - v;
}

// `cnt` holds, for every wave w and digit b < nbins, the number of the wave's
// items with digit b at cnt[w * stride + b] (u16, filled by rank_round).
// On return:
//   cnt[w * stride + b] = items with digit b in waves before w,
//   excl[b]             = items of the block with digit < b (b <= nbins).
// Together with rank_round's per-wave rank this gives every item its stable
// position in the block's digit-sorted order.
template <int NT>
__device__ void block_digit_offsets(uint16_t* cnt, int stride, int nbins,
                                    uint32_t* excl, uint32_t* scratch) {
  constexpr int NW = NT / kWave;
  const int per = (nbins + NT - 1) / NT;
  const int b0 = threadIdx.x * per;
  uint32_t local = 0;
  for (int i = 0; i < per; ++i) {
    const int b = b0 + i;
    if (b < nbins) {
      uint32_t s = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const uint32_t c = cnt[w * stride + b];
        cnt[w * stride + b] = (uint16_t)s;
        s += c;
      }
      excl[b] = s;  // bin total for now
      local += s;
    }
  }
  uint32_t total;
  uint32_t run = block_excl_scan_u32<NT>(local, scratch, total);
  for (int i = 0; i < per; ++i) {
    const int b = b0 + i;
    if (b < nbins) {
      const uint32_t c = excl[b];
      excl[b] = run;
      run += c;
    }
  }
  if (threadIdx.x == 0) excl[nbins] = total;
  block_sync();
}

}  // namespace semsched
