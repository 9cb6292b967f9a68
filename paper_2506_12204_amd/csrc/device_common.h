// Device helpers shared by the gfx950 scheduling kernels: wave64 digit
// matching and ranking, wave-level scans and reductions, exact 128-bit
// accumulation. Nothing here is specific to one kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace semsched {

constexpr int kWave = 64;

// Integer types that may alias any other type. LDS buffers are reused with
// different element widths (u16 counters in a u64 stage, u16 counters cleared
// a u64 at a time, two u16 counters read as one u32); accesses through these
// types keep the compiler from reordering them past accesses of the other
// width, which strict aliasing would otherwise allow.
typedef uint64_t __attribute__((may_alias)) u64_alias;
typedef uint32_t __attribute__((may_alias)) u32_alias;
typedef uint16_t __attribute__((may_alias)) u16_alias;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Workgroup barrier that first drains this wave's outstanding LDS operations.
// __syncthreads() alone may let a wave reach s_barrier with LDS loads still in
// flight; another wave can then overwrite the location after the barrier
// before that load has read it (observed as corrupted elements when the wave
// counters reuse the stage buffer). Every barrier in these kernels guards a
// write-after-read or read-after-write hand-over of LDS, so all of them wait.
__device__ __forceinline__ void block_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __syncthreads();
}

__device__ __forceinline__ uint32_t bit_width32(uint32_t x) {
  return x ? 32u - __clz(x) : 0u;
}

__device__ __forceinline__ uint64_t lanes_below() { return __lanemask_lt(); }

// Mask of the lanes of the wave whose `d` agrees with this lane's on the low
// `nbits` bits. Every lane of the wave must execute it (all 64 are active in
// every caller: invalid items carry a sentinel digit instead of idling).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, int nbits) {
  uint64_t peers = ~0ull;
#pragma unroll
  for (int b = 0; b < 10; ++b) {  // digits have at most 10 bits
    if (b < nbits) {
      const bool set = (d >> b) & 1u;
      const uint64_t m = __ballot(set);
      peers &= set ? m : ~m;
    }
  }
  return peers;
}

// Stable per-wave ranking of one round of 64 digits against this wave's
// running counters `cnt` (LDS, one u16 per digit, private to the wave).
// Returns the number of earlier items of the wave (earlier rounds, then lower
// lanes of this round) that carry the same digit, and advances the counter.
__device__ __forceinline__ uint32_t rank_round(uint32_t d, int nbits,
                                               uint16_t* cnt) {
  const uint64_t peers = match_digit(d, nbits);
  const uint32_t below = __popcll(peers & lanes_below());
  const uint32_t base = cnt[d];
  // All peers have read the old count before the lowest peer writes the new
  // one: a wave's LDS operations complete in program order.
  if (below == 0) cnt[d] = (uint16_t)(base + __popcll(peers));
  return base + below;
}

// The lanes of the wave whose digit differs from this lane's in at least one
// of the low NB bits (NB known at compile time). Per bit: the lane's bit as a
// 0/-1 mask, its ballot, and one three-input bit operation per half that ORs
// (ballot XOR mask) -- the lanes whose bit differs -- into the set. Four VALU
// operations per bit. The empty asm keeps the compiler from recomputing the
// ballot's predicate by other means.
template <int NB>
__device__ __forceinline__ uint64_t mismatch_digit_c(uint32_t d) {
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)d, b, 1);
    asm("" : "+v"(m));
    const uint64_t bal = __builtin_amdgcn_ballot_w64(m != 0);
    // 0xF6 = A | (B ^ C) for sources (A, B, C)
    lo = __builtin_amdgcn_bitop3_b32(lo, (uint32_t)bal, m, 0xF6);
    hi = __builtin_amdgcn_bitop3_b32(hi, (uint32_t)(bal >> 32), m, 0xF6);
  }
  return ((uint64_t)hi << 32) | lo;
}

// The lanes with the same digit as this lane (match_digit for a compile-time
// width).
template <int NB>
__device__ __forceinline__ uint64_t match_digit_c(uint32_t d) {
  return ~mismatch_digit_c<NB>(d);
}

// rank_round for a compile-time digit width. Every peer writes the same new
// count, so no lane has to be singled out for the update. The peers and the
// other lanes split the wave, so the peers below this lane are the lanes
// below it minus the mismatching ones below it, and the peers number 64 minus
// the mismatching lanes.
template <int NB>
__device__ __forceinline__ uint32_t rank_round_c(uint32_t d, uint16_t* cnt) {
  const uint64_t other = mismatch_digit_c<NB>(d);
  const uint32_t below = (uint32_t)lane_id() - __builtin_amdgcn_mbcnt_hi(
      (uint32_t)(other >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)other, 0u));
  const uint32_t base = cnt[d];
  cnt[d] = (uint16_t)(base + (uint32_t)kWave - (uint32_t)__popcll(other));
  uint32_t rank = base + below;
  // settle the rank now: left to itself the compiler keeps the count, the
  // peer mask and the address of every round alive until their last use
  asm volatile("" : "+v"(rank));
  return rank;
}

// Stable per-wave ranking of one round by digit through a table of 64-bit
// lane masks in LDS, one per digit, private to the wave and zero on entry and
// on return. Every lane ORs its bit into its digit's mask, reads the mask
// back (its peers: a wave's LDS operations complete in program order, so all
// of the round's bits are in) and clears it again. Three LDS operations and
// a few VALU ones, where matching the digit bit by bit with ballots takes
// four VALU operations per bit. Returns, as rank_round_c, the number of
// earlier items of the wave with the same digit and advances the counter.
__device__ __forceinline__ uint32_t rank_round_mask(uint32_t d, u64_alias* masks,
                                                    uint16_t* cnt) {
  // Each half of the wave sets and clears only its own 32-bit half of the
  // digit's mask (one bank per lane instead of two); the peers are read as
  // the whole 64-bit mask.
  const uint32_t lane = (uint32_t)lane_id();
  u32_alias* half = reinterpret_cast<u32_alias*>(masks + d) + (lane >> 5);
  atomicOr(reinterpret_cast<unsigned int*>(half), 1u << (lane & 31u));
  const uint64_t peers = masks[d];
  *half = 0;
  const uint32_t below = __builtin_amdgcn_mbcnt_hi(
      (uint32_t)(peers >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u));
  const uint32_t base = cnt[d];
  cnt[d] = (uint16_t)(base + (uint32_t)__popcll(peers));
  uint32_t rank = base + below;
  asm volatile("" : "+v"(rank));
  return rank;
}

// Zeroes NBIN u64 entries (a wave's mask table) with this wave's lanes.
template <int NBIN>
__device__ __forceinline__ void clear_wave_masks(u64_alias* masks) {
  static_assert(NBIN % kWave == 0, "whole rounds of lanes");
#pragma unroll
  for (int i = 0; i < NBIN / kWave; ++i) masks[i * kWave + lane_id()] = 0;
}

// Hides a value's origin from the optimiser, so that an address derived from
// it is recomputed after a barrier instead of being kept in a register.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Inclusive scan of a 32-bit value over the wave with DPP lane moves: four
// row_shr steps scan each row of 16 lanes, then row_bcast:15 and
// row_bcast:31 carry the row totals into the rows above. Lanes whose source
// is outside the row (or whose row is masked off) add 0.
__device__ __forceinline__ uint32_t wave_incl_scan_dpp(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

// Exact inclusive wave scan of 32-bit values (lengths) into 64 bits: the low
// and high 16-bit halves are scanned separately, each sum staying below 2^22.
__device__ __forceinline__ uint64_t wave_incl_scan_len(uint32_t v) {
  const uint32_t lo = wave_incl_scan_dpp(v & 0xffffu);
  const uint32_t hi = wave_incl_scan_dpp(v >> 16);
  return ((uint64_t)hi << 16) + lo;
}

// Exact inclusive wave scan of values below 2^40 (per-thread sums of a few
// bins' length totals): two 20-bit parts, each sum staying below 2^26.
__device__ __forceinline__ uint64_t wave_incl_scan_u40(uint64_t v) {
  const uint32_t lo = wave_incl_scan_dpp((uint32_t)v & 0xfffffu);
  const uint32_t hi = wave_incl_scan_dpp((uint32_t)(v >> 20));
  return ((uint64_t)hi << 20) + lo;
}

// Value of lane 63 (the wave total after an inclusive scan).
__device__ __forceinline__ uint64_t last_lane_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive wave scan of a 64-bit value.
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint64_t o = __shfl_up(v, off, kWave);
    if (lane_id() >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) { return wave_incl_scan_dpp(v); }

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v = min(v, (uint32_t)__shfl_xor(v, off, kWave));
  return v;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor(v, off, kWave));
  return v;
}

__device__ __forceinline__ uint32_t wave_or_u32(uint32_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v |= (uint32_t)__shfl_xor(v, off, kWave);
  return v;
}

// Unsigned 128-bit accumulator (waits are non-negative).
struct U128 {
  uint64_t lo, hi;
};

__device__ __forceinline__ void add128(U128& a, uint64_t v) {
  a.lo += v;
  a.hi += (a.lo < v) ? 1u : 0u;
}

__device__ __forceinline__ void add128(U128& a, const U128& b) {
  a.lo += b.lo;
  a.hi += b.hi + ((a.lo < b.lo) ? 1u : 0u);
}

// Wave-wide sum of 128-bit values (result valid in every lane).
__device__ __forceinline__ U128 wave_sum128(U128 v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    U128 o;
    o.lo = __shfl_xor(v.lo, off, kWave);
    o.hi = __shfl_xor(v.hi, off, kWave);
    add128(v, o);
  }
  return v;
}

// Atomically add a 128-bit value into (lo, hi) words. The carry out of the
// low word is derived from the value it held just before this addition, so
// the pair stays exact under any interleaving of such calls.
__device__ __forceinline__ void atomic_add128(uint64_t* lo, uint64_t* hi,
                                              const U128& v) {
  const uint64_t old =
      atomicAdd(reinterpret_cast<unsigned long long*>(lo), (unsigned long long)v.lo);
  const uint64_t carry = (old + v.lo < old) ? 1u : 0u;
  atomicAdd(reinterpret_cast<unsigned long long*>(hi),
            (unsigned long long)(v.hi + carry));
}

// Relaxed agent-scope load of a word other workgroups (possibly on other
// XCDs) update with atomics, such as the error flags: coherent across the
// XCDs' L2 caches, with no ordering against other memory.
template <typename T>
__device__ __forceinline__ T load_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace semsched
