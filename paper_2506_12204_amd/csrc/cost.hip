// Cost model of Section 3.4: remaining computation time of every request
// (the f_t the scheduler orders by within an urgency level) and the cache /
// recompute decisions of an eviction.
//
// Constants are Q32.32 integers (time unit x 2^32 per token, or per token^2
// for alpha1); every product is formed exactly in 128 bits:
//
//   prefill(n)   = alpha1 * n^2 + alpha2 * n
//   decode(n, m) = gamma1 * ((m^2 + m) / 2 + n * m) + gamma2 * m      (Eq. 4:
//                  tokens n+1 .. n+m at gamma1 * i + gamma2 each)
//   service      = floor(cost / 2^32) saturated at 2^31 - 1, with cost =
//                  decode(n + d, max(m - d, 0)) + (d == 0 ? prefill(n) : 0)
//                  for prompt n, predicted output m, d tokens decoded so far
//   keep         = beta * n < prefill(n)   (Eq. 3 with the comparison its
//                  text explains: keep the cache when reloading is cheaper)
//   save         = m' - y*, y* the first y in [0, m'] with
//                  gamma1 * (y + 1 + n) + gamma2 >= beta (the integer
//                  minimiser of Eq. 5, the largest saved count among ties)
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace semsched {

namespace {

constexpr int CT = 256;
constexpr int kCostBlocks = 2048;

__device__ __forceinline__ U128 mul64(uint64_t a, uint64_t b) { return {a * b, __umul64hi(a, b)}; }

// a += b, recording a carry out of 128 bits in `over`.
__device__ __forceinline__ void add_sat(U128& a, const U128& b, bool& over) {
  const uint64_t lo = a.lo + b.lo;
  const uint64_t c = lo < b.lo ? 1u : 0u;
  const uint64_t hi = a.hi + b.hi + c;
  over |= hi < a.hi || (hi == a.hi && (b.hi | c) != 0);
  a = {lo, hi};
}

__device__ __forceinline__ int32_t service_of(const CostArgs& a, uint64_t n, uint64_t m,
                                              uint64_t d) {
  const uint64_t r = m > d ? m - d : 0;
  bool over = false;
  U128 cost = mul64(a.gamma1, (r * r + r) / 2 + (n + d) * r);  // (< 2^61 + 2^63)
  add_sat(cost, mul64(a.gamma2, r), over);
  if (d == 0) {
    add_sat(cost, mul64(a.alpha1, n * n), over);
    add_sat(cost, mul64(a.alpha2, n), over);
  }
  // floor(cost / 2^32), saturated
  if (over || (cost.hi >> 32) != 0) return INT32_MAX;
  const uint64_t s = (cost.hi << 32) | (cost.lo >> 32);
  return s > (uint64_t)INT32_MAX ? INT32_MAX : (int32_t)s;
}

__device__ __forceinline__ void flag_range(uint32_t* flags, bool bad) {
  if (__ballot(bad) && lane_id() == 0) atomicOr(flags, kFlagRange);
}

__global__ __launch_bounds__(CT) void c_service(CostArgs a) {
  const int64_t stride = (int64_t)gridDim.x * CT;
  for (int64_t i0 = (int64_t)blockIdx.x * CT; i0 < a.n; i0 += stride) {
    const int64_t i = i0 + threadIdx.x;
    const bool live = i < a.n;
    const int64_t ic = live ? i : a.n - 1;
    const int32_t n = a.prompt[ic], m = a.output[ic];
    const int32_t d = a.decoded ? a.decoded[ic] : 0;
    const bool bad = live && (n < 0 || m < 0 || d < 0);
    flag_range(a.flags, bad);
    if (live) {
      a.service[i] = bad ? 0
                         : service_of(a, (uint64_t)n, (uint64_t)m, (uint64_t)d);
    }
  }
}

__global__ __launch_bounds__(CT) void c_evict(CostArgs a) {
  const int64_t stride = (int64_t)gridDim.x * CT;
  for (int64_t i0 = (int64_t)blockIdx.x * CT; i0 < a.n; i0 += stride) {
    const int64_t i = i0 + threadIdx.x;
    const bool live = i < a.n;
    const int64_t ic = live ? i : a.n - 1;
    const int32_t n = a.prompt[ic], mp = a.decoded[ic];
    const bool bad = live && (n < 0 || mp < 0);
    flag_range(a.flags, bad);
    if (!live) continue;
    if (bad) {
      a.keep[i] = 0;
      a.save[i] = 0;
      continue;
    }
    const uint64_t un = (uint64_t)n;
    // keep the prefill cache when reloading (beta * n) is cheaper than recomputing
    const U128 reload = mul64(a.beta, un);
    bool over = false;
    U128 recompute = mul64(a.alpha1, un * un);
    add_sat(recompute, mul64(a.alpha2, un), over);
    const bool keep = over || reload.hi < recompute.hi ||
                      (reload.hi == recompute.hi && reload.lo < recompute.lo);
    a.keep[i] = keep ? 1 : 0;
    // first y whose next recomputed token does not pay
    int64_t y;
    if (a.gamma2 >= a.beta) {
      y = 0;
    } else if (a.gamma1 == 0) {
      y = mp;
    } else {
      const uint64_t t = a.beta - a.gamma2;
      const uint64_t q = t / a.gamma1 + (t % a.gamma1 != 0 ? 1u : 0u);  // ceil(t / gamma1)
      const int64_t v = (int64_t)q - 1 - (int64_t)un;                     // (q < 2^64 / 1)
      y = q > (uint64_t)INT64_MAX ? (int64_t)mp : max(v, (int64_t)0);
      y = min(y, (int64_t)mp);
    }
    a.save[i] = (int32_t)(mp - y);
  }
}

// The scheduler resets the error word when it starts; the cost pass's range
// errors are kept in a word of their own and added afterwards.
__global__ void c_merge_flags(uint32_t* dst, const uint32_t* src) {
  if (threadIdx.x == 0 && *src) atomicOr(dst, *src);
}

int grid_for(int64_t n) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((n + CT - 1) / CT, kCostBlocks));
}

}  // namespace

hipError_t launch_service(const CostArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after) {
  if (before) (void)hipEventRecord(before, st);
  if (a.n > 0) hipLaunchKernelGGL(c_service, dim3(grid_for(a.n)), dim3(CT), 0, st, a);
  if (after) (void)hipEventRecord(after, st);
  return hipGetLastError();
}

hipError_t launch_evict(const CostArgs& a, hipStream_t st) {
  if (a.n > 0) hipLaunchKernelGGL(c_evict, dim3(grid_for(a.n)), dim3(CT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_merge_flags(uint32_t* dst, const uint32_t* src, hipStream_t st) {
  hipLaunchKernelGGL(c_merge_flags, dim3(1), dim3(64), 0, st, dst, src);
  return hipGetLastError();
}

}  // namespace semsched
