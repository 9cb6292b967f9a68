// Host/device interface of the scheduling kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace semsched {

// Device-detected error bits, OR-ed into the workspace's first word.
constexpr uint32_t kFlagInval = 1u;  // bad offsets / queue longer than promised
constexpr uint32_t kFlagRange = 2u;  // length < 0 or priority >= num_classes
constexpr uint32_t kFlagDevice = 4u; // an internal consistency check failed on the device

// ---------------------------------------------------------------------------
// Queues scheduled inside one workgroup's LDS (batched.hip).
//
// Size classes of the batched call. A queue of at most kSegTinyCap requests
// is scheduled by one wave; up to kSegMediumCap by a 256-thread workgroup;
// up to kSegLargeCap (and every shorter queue whose key does not fit a
// 32-bit element) by a 512-thread workgroup on 64-bit elements; longer
// queues by the multi-workgroup segmented sort.
constexpr int kSegTinyCap = 256;
constexpr int kSegMediumCap = 4096;
constexpr int kSegLargeCap = 16384;
constexpr int kLongTile = 8192;   // requests per tile of the segmented sort

// Work lists of the batched call, one per kernel.
enum BList { kListTiny = 0, kListMedium = 1, kListWide = 2, kListLong = 3, kLists = 4 };
constexpr int kSubLists = 8;      // the medium and wide lists: 8 segments each
constexpr int kPlanChunk = 256;   // most queues the planner files per chunk

// The medium and wide lists are kept in kSubLists segments: segment j holds
// the queues of the planner's chunks c with c % kSubLists == j (and the
// queues of those chunks handed on), so that the planner's filing atomics
// spread over kSubLists counters. A segment holds at most ceil(S / 8) +
// kPlanChunk queues for S queues and chunks of at most kPlanChunk.
inline int64_t list_segment_cap(int64_t num_segments) {
  return (num_segments + kSubLists - 1) / kSubLists + kPlanChunk;
}

// Per-call control block at the start of a batched workspace (after the
// 64-byte flags line), followed by the segment lines.
struct BCtl {
  uint32_t count[kLists];             // entries of the long list (count[kListLong])
  uint32_t empty[kLists][kSubLists];  // 1 once a segment was found exhausted (a hint)
  uint64_t long_elems;                // requests in the long list's queues
  uint32_t ranges[5];                 // long queues: pmin, pmax, lmin, lmax, longest
};
// One segment of a list, alone in its 128-byte line: its entry count (the
// planner's filing atomics) and the next batch to grab (the kernels'
// atomics). Atomics on one line are serialised wherever they come from, so
// counters that shared a line would be one counter.
struct alignas(128) GrabLine {
  uint32_t next;
  uint32_t count;
  uint32_t pad[30];
};

// One tile of the segmented sort of the long queues: found once per call by a
// search over the queues' first tiles, then read by every later phase with
// one load.
struct LongTileDesc {
  int64_t first;   // global index of the tile's first request
  uint64_t at;     // position of that request in the keys/ids arrays
  int64_t s;       // the queue
  uint32_t lo;     // the tile's first request within the queue
  int32_t cnt;     // requests in the tile
  uint32_t item0;  // the queue's first digit-offset work item
  uint32_t rows;   // tiles of the queue
};

struct BArgs {
  const uint8_t* priority;
  const int32_t* length;
  const int64_t* offsets;   // [num_segments + 1]; null: one queue of n_single requests
  int64_t num_segments;
  int64_t n_single;
  int32_t num_classes;      // validation bound and totals stride - 1
  int32_t* order;
  int64_t* wait;
  uint64_t* totals;         // (lo, hi) pairs, num_segments * (1 + num_classes)
  uint32_t* flags;
  BCtl* ctl;
  GrabLine* grab;           // [kLists][kSubLists]
  // queue indices: the medium list's kSubLists segments of seg_cap entries,
  // the wide list's, then the long list's num_segments entries
  uint32_t* lists;
  int64_t seg_cap;          // list_segment_cap(num_segments)
  // segmented sort of the long queues (capacity: requests in long queues)
  uint64_t long_cap;
  uint32_t max_tiles;
  uint64_t* keys[2];        // [long_cap]
  uint32_t* ids[2];         // [long_cap]
  uint32_t* hist;           // [max_tiles][2^kLongDigitBits] digit counts, then offsets
  uint64_t* tsum;           // [max_tiles] length sums, then wait bases
  uint64_t* lbase;          // [long list + 1] start of every long queue in keys/ids
  uint32_t* tstart;         // [long list + 1] first tile of every long queue
  uint32_t* istart;         // [long list + 1] first digit-offset work item of every long queue
  uint32_t* qtot;           // [kLongColDigits * long_items_max] digit totals of the queues of many tiles
  LongTileDesc* tdesc;      // [max_tiles] every tile's place, written once per call
  uint32_t* imap;           // [long_items_max] first tile of each digit-offset item's queue
};

// Single queue of a.n_single <= kSegLargeCap requests (a.offsets null), one
// workgroup, any key width.
hipError_t launch_single_lds(const BArgs& a, hipStream_t st);
// The whole batched schedule: planner, the LDS kernels of every size class,
// the segmented sort of long queues. a.flags and a.ctl zeroed by the caller.
hipError_t launch_batched(const BArgs& a, hipStream_t st);
// Workspace parts of the segmented sort for `long_cap` requests in long
// queues out of num_segments queues.
uint32_t long_max_tiles(uint64_t long_cap, int64_t num_segments);
// Digits of a pass of the segmented sort of the long queues.
constexpr int kLongDigitBits = 10;
// A long queue of at most kLongRowsFew tiles takes its digit offsets in one
// work item; a longer one in one per kLongColDigits digits.
constexpr uint32_t kLongRowsFew = 32;
// Digits of one work item of a longer queue (its columns are scanned together).
constexpr int kLongColDigits = 16;
// Most digit-offset work items of the long queues.
inline uint64_t long_items_max(uint64_t long_cap, int64_t queues) {
  return (uint64_t)queues + ((1u << kLongDigitBits) / kLongColDigits) *
                                (long_cap / ((uint64_t)kLongRowsFew * kLongTile) + 1);
}

// ---------------------------------------------------------------------------
// Global multi-pass path (one queue longer than kSegLargeCap).

constexpr int kMaxBins = 1024;   // digit bins of every scatter pass
constexpr int kMaxScatter = 5;   // scatter passes: first, up to 3 middle, final
constexpr int kGlobalThreads = 512;
constexpr int kGlobalRounds = 8;
constexpr int kGlobalTile = kGlobalThreads * kGlobalRounds;
constexpr int kFirstTiles = 4;   // the first pass works on 4 tiles at a time
// Histogram rows per block of the first and final passes (a row is counted
// by a workgroup of its own; a block's offsets are the column scan at its
// first row). More rows did not speed the histograms up and slowed the column
// scans, so each block is one row.
constexpr int kHistRows = 1;
static_assert(kFirstTiles % kHistRows == 0, "a block splits into whole-tile rows");
constexpr int kMaxBlocks = 4096; // upper bound on workgroups of a pass

// Compact two-pass layout. Between the passes an element is one u32: the
// final digit above the low kChunkBits bits of the request id. The id's high
// bits (its chunk, id >> kChunkBits) and the first digit are not stored: the
// first pass leaves every first-digit bucket in id order, so an element's
// bucket and chunk follow from its position and the sub-bucket starts
// (bucket, chunk) counted by the histogram pass.
constexpr int kChunkBits = 22;
constexpr int kMaxChunks = 256;  // ids below 2^30

// Decided on the device by the histogram pass once the ranges are known.
struct Plan {
  uint32_t ok;        // 0 if a range error was found, or the middle passes'
                      // grid barrier gave up
  uint32_t pmin;      // smallest priority
  uint32_t hmin;      // smallest length >> d0
  uint32_t H;         // (largest length >> d0) - hmin + 1
  uint32_t P;         // largest priority - pmin + 1
  uint32_t wh, wp;    // bit widths of the h and p fields of a key
  uint32_t W;         // bits below the key in a packed element: 32 when the
                      // key fits 32 bits (key in the high word), else the
                      // bit width of a request id
  uint32_t packed;    // 1: element = key << W | id in one u64
  uint32_t small;     // 1: every length < 2^26 (64-lane length sums fit 32 bits)
  uint32_t nscatter;  // number of scatter passes (>= 2)
  uint32_t compact;   // 1: the compact two-pass layout (u32 elements) is used
  uint32_t pay;       // 1: compact elements also carry the caller's rank above the
                      // final digit (the rank takes no part in the order)
  uint32_t pay_shift; // bit of a compact element where that rank starts
  uint32_t cglb;      // compact: 1 if some block of the final pass needs the
                      // global-window kernel (sub-bucket starts beyond the LDS
                      // window, or a queue too long for buffer-resource stores)
  uint32_t shift[kMaxScatter];  // digit = (u2 >> shift) & (bins - 1), passes >= 1
  uint32_t nbits[kMaxScatter];
  uint32_t nbins[kMaxScatter];
};

// Grid barrier of the middle-pass kernel: the arrival count and the release
// word in lines of their own, so that polling the one does not slow the
// atomics on the other.
struct MidSync {
  alignas(128) uint32_t arrive;
  alignas(128) uint32_t release;
};

// A pass's work split: workgroup g owns tiles [g*tpb, min(tiles, (g+1)*tpb)).
struct Split {
  int32_t blocks;
  int32_t tpb;
};

struct GArgs {
  const uint8_t* priority;
  const int32_t* length;
  int64_t n;
  int32_t* order;
  int64_t* wait;
  uint64_t* totals;     // (lo, hi) pairs, 1 + num_classes
  int32_t num_classes;
  int32_t d0;           // width of the first (low-length) digit
  int32_t tiles;
  int32_t force_wide;   // 1: never pack the id into the key word
  int32_t chunked;      // 1: the histogram pass counts the chunk sub-buckets, so the
                        // compact layout may be chosen (host: kchunks <= kMaxChunks,
                        // blocks of the first pass no longer than a chunk)
  int32_t kchunks;      // K = ceil(n / 2^kChunkBits) id chunks
  int32_t kpb;          // log2 of Kp, the power of two >= K that strides sub_start
  Split main;           // first histogram and first pass (tpb a multiple of kFirstTiles)
  Split fin;            // final histogram and final pass
  Split mid;            // the middle-pass kernel (its grid: the resident-workgroup limit)
  int32_t split_mid;    // 1: the middle passes run as separate launches per phase
  uint32_t mid_spin;    // polls of the middle-pass grid barrier before it gives up
  MidSync* msync;       // that barrier's state
  uint32_t* flags;
  uint64_t* sink;       // 16 bytes that absorb the stores of lanes without an item
                        // (so that a pass's stores are unconditional)
  uint32_t* block_ranges;  // [blocks][4] pmin, pmax, lmin, lmax of every block
  Plan* plan;
  uint32_t* hist_cnt;   // [kMaxScatter][kMaxBins] digit totals of every pass
  uint64_t* hist_w;     // [kMaxBins] length sums of the final digit
  uint32_t* block_hist; // [blocks][kMaxBins] digit counts per block, then offsets
  uint64_t* block_histw;// [blocks][kMaxBins] final-digit length sums, then offsets
  uint64_t* keys[2];
  uint32_t* ids[2];
  uint32_t* chunk_part; // [kMaxChunks][kMaxBins] first-digit counts of the ids of
                        // chunk boundary k's block that lie below the boundary
  uint32_t* sub_start;  // [kMaxBins][Kp] start of sub-bucket (digit d, chunk k)
                        // relative to bucket d's start; k >= K hold the bucket size
  // Optional (SJF): ranks carried through the sort but not ordered by, and
  // their largest value (written by an earlier kernel). When the compact
  // layout has room for them, the final pass splits the totals by these
  // ranks instead of by `priority`.
  const uint8_t* payload;
  const uint32_t* pay_pmax;
};

// Optional events recorded around one stage's kernel (null: not armed).
constexpr int kStages = 7;  // hist, first, final (long queues); merge; policy; cost; middle passes
struct StageEvents {
  hipEvent_t before[kStages];
  hipEvent_t after[kStages];
};

// Work splits of the passes for n requests (device-dependent occupancy).
Split global_first_split(int64_t n);
Split global_final_split(int64_t n);
Split global_mid_split(int64_t n);
hipError_t launch_global_schedule(const GArgs& a, hipStream_t st, const StageEvents* ev);

// Zeroes `count` 32-bit words (graph-safe replacement for a memset).
hipError_t launch_fill_zero(uint32_t* p, size_t count, hipStream_t st);

// ---------------------------------------------------------------------------
// Insertion of arrivals into an existing schedule (insert.hip).
constexpr int kInsUnit = 1024;  // earlier entries per unit of the merge pass (one wave)

struct InsArgs {
  const uint8_t* priority;  // [n_old + m], earlier requests first
  const int32_t* length;
  int64_t n_old, m;
  const int32_t* order_old; // [n_old] the earlier schedule
  const int64_t* wait_old;
  const int32_t* order_m;   // [m] the arrivals' own schedule (ids local to them)
  const int64_t* wait_m;
  uint32_t* ins;            // [max(m, 1)] earlier entries not above each arrival
  uint64_t* desc;           // [units + 1] per unit of kInsUnit earlier entries: arrivals
                            // placed before its first entry (bits 0..31), the class of
                            // its first (32..39) and of its last entry (40..47)
  uint32_t* cs;             // [257] class starts of the earlier sequence
  uint64_t* lsum;           // [2] total lengths of the two sequences
  uint64_t* sink;           // 16 bytes that absorb the stores of lanes without an entry
  int32_t* order;           // [n_old + m] the merged schedule
  int64_t* wait;
  uint64_t* totals;         // (lo, hi) pairs, 1 + 256, zeroed by the caller
};

// Units of kInsUnit earlier entries (desc holds one more entry).
int64_t insert_units(int64_t n_old);
// `before` / `after` (may be null) are recorded around the merge kernel.
hipError_t launch_insert(const InsArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after);

// ---------------------------------------------------------------------------
// Comparison policies (policy.hip): FCFS, SJF's class totals, HPJF.
constexpr int kPolRange = 4096;  // positions per wave of the policy kernels

struct PolArgs {
  const uint8_t* priority;  // [n]
  const int32_t* length;    // [n]
  int64_t n;
  int32_t* order;           // [n] (SJF: the schedule already computed)
  int64_t* wait;            // [n]
  uint64_t* totals;         // (lo, hi) pairs, 1 + 256, zeroed by the caller (FCFS, HPJF)
  uint32_t* flags;          // device error bits
  uint32_t* pmax;           // largest rank, zeroed by the caller
  uint64_t* rsum;           // [ranges] FCFS: length sum per range, then range offsets
  uint32_t* tab_cnt;        // [ranges * P] HPJF: per range and class, count, then offset
  uint64_t* tab_len;        // [ranges * P] HPJF: per range and class, length sum, then offset
  uint32_t* ctot_cnt;       // [256] HPJF: class sizes
  uint64_t* ctot_len;       // [256] HPJF: class length totals
  uint64_t* part;           // [blocks * P] (lo, hi) per-block class sums
  uint64_t* sink;           // 16 bytes for the stores of lanes without an element
  const uint32_t* pay;      // SJF: nonzero once the sort split the totals by rank itself
                            // (the plan's flag; null when the sort has no plan)
};

int64_t policy_ranges(int64_t n);
int64_t policy_blocks(int64_t n);
// `before` / `after` (may be null) are recorded around the pass that writes
// the schedule (FCFS, HPJF) or sums the classes (SJF).
hipError_t launch_fcfs(const PolArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after);
hipError_t launch_hpjf(const PolArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after);
// Largest rank of a.priority into a.pmax (zeroed by the caller).
hipError_t launch_policy_range(const PolArgs& a, hipStream_t st);
// SJF's class sums after the sort; the caller ran launch_policy_range.
hipError_t launch_class_totals(const PolArgs& a, hipStream_t st, hipEvent_t before,
                               hipEvent_t after);

// ---------------------------------------------------------------------------
// Cost model (cost.hip).
struct CostArgs {
  const int32_t* prompt;   // [n] prompt tokens
  const int32_t* output;   // [n] predicted output tokens (service times only)
  const int32_t* decoded;  // [n] tokens decoded so far (null: all 0)
  int64_t n;
  uint64_t alpha1, alpha2, beta, gamma1, gamma2;  // Q32.32
  int32_t* service;        // [n] out: remaining computation time
  uint8_t* keep;           // [n] out: 1 = keep the prefill cache of an eviction
  int32_t* save;           // [n] out: decoded tokens whose cache is saved
  uint32_t* flags;         // device error bits
};

hipError_t launch_service(const CostArgs& a, hipStream_t st, hipEvent_t before, hipEvent_t after);
hipError_t launch_evict(const CostArgs& a, hipStream_t st);
hipError_t launch_merge_flags(uint32_t* dst, const uint32_t* src, hipStream_t st);

// ---------------------------------------------------------------------------
// Batch selection and eviction (batch.hip): one workgroup over LDS up to
// these sizes, several kernels over the workspace beyond them.
constexpr int kSelectCap = 4096;  // largest batch, buffer and ongoing set in LDS
constexpr int kEvictCap = 8192;   // most cached requests in LDS
constexpr int kWideChunk = 8192;  // entries sorted by one workgroup beyond those
constexpr int64_t kWideMax = 1ll << 30;  // entries of all lists of one call

struct SelArgs {
  const uint8_t* priority;  // [n_ids]
  const int32_t* length;    // [n_ids]
  const uint8_t* stage;     // [n_ids] 0 = prefill, 1 = decoding
  int64_t n_ids;
  const int32_t* heap_order;  // [n_heap] the waiting requests' schedule (first b read)
  int64_t n_heap;
  const int32_t* buffer;    // [n_buffer] arrivals not yet in the schedule
  int64_t n_buffer;
  const int32_t* ongoing;   // [n_ongoing]
  int64_t n_ongoing;
  int64_t b;
  int32_t* batch;           // [b]
  int32_t* pushed;          // [b + n_ongoing]
  int64_t* counts;          // [2] batch size, pushed-back count
  uint32_t* flags;
};

struct EvictArgs {
  const uint8_t* priority;
  const int32_t* length;
  int64_t n_ids;
  const int32_t* cached;    // [n_cached]
  const int64_t* kv;        // [n_cached] KV size of each cached request
  int64_t n_cached;
  int64_t usage, capacity;
  const int64_t* demands;   // [n_demands] KV demand of each incoming request
  int64_t n_demands;
  int32_t* victims;         // [n_cached] eviction order, first upto[last] written
  int64_t* upto;            // [n_demands] victims after each incoming request
  uint32_t* flags;
};

// A list of request ids to sort by key: src0[0 .. n0) then src1[0 .. n1),
// placed at entries [base, base + n0 + n1) of the sort arrays.
struct WideList {
  const int32_t* src0;
  int64_t n0;
  const int32_t* src1;
  int64_t n1;
  int64_t base;
};

// The sort of up to two lists beyond one workgroup's LDS: (key, id) entries
// (and, for eviction, the index into the caller's arrays) in two buffers that
// the chunk sort and the merge rounds ping-pong between.
struct WideSort {
  const uint8_t* priority;
  const int32_t* length;
  int64_t n_ids;
  const int64_t* kv;  // eviction: KV sizes, checked for >= 0; else null
  WideList list[2];
  int32_t nlists;
  int64_t total;      // entries of all lists
  uint64_t* key[2];
  uint32_t* id[2];
  uint32_t* pay[2];   // eviction only
  uint32_t* flags;
};

hipError_t launch_select(const SelArgs& a, hipStream_t st);
hipError_t launch_evict_victims(const EvictArgs& a, hipStream_t st);
// Beyond the LDS sizes: w holds the lists (candidates, then ongoing; or the
// cached requests) and the sort buffers; dec [candidates + 1] u32, psum
// [n_cached] u64 and eorder [n_cached] u32 are workspace arrays.
hipError_t launch_select_wide(const SelArgs& a, WideSort w, uint32_t* dec, hipStream_t st);
hipError_t launch_evict_wide(const EvictArgs& a, WideSort w, uint64_t* psum, uint32_t* eorder,
                             hipStream_t st);

}  // namespace semsched
