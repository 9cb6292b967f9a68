// C ABI of the scheduling library: argument checks, workspace layout, launch
// planning and error mapping. The operations themselves are defined in
// semsched.h; every step of them runs in the HIP kernels of this directory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "kernels.h"
#include "semsched.h"

using namespace semsched;

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kHeaderBytes = 256;  // flags, counters, ranges, plan

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  size_t flags = 0, sink = 16, plan = 64;
  size_t hist_cnt = 0, hist_w = 0, block_hist = 0, block_histw = 0, block_ranges = 0;
  size_t keys0 = 0, keys1 = 0, ids0 = 0, ids1 = 0, chunk_part = 0, sub_start = 0, msync = 0;
  size_t total = kHeaderBytes;
  int64_t tiles = 0;
};

static_assert(sizeof(Plan) <= kHeaderBytes - 64, "plan must fit in the header");

bool needs_global(int64_t n) { return n > kSegLargeCap; }

// Sizes depend on n only (not on the device), so the workspace size can be
// asked for anywhere.
Layout layout_for(int64_t n) {
  Layout L;
  if (!needs_global(n)) return L;
  L.tiles = (n + kGlobalTile - 1) / kGlobalTile;
  // histogram rows: whole blocks of kHistRows rows, never more than kMaxBlocks
  const size_t blocks = (size_t)std::min<int64_t>(
      (L.tiles + kHistRows - 1) / kHistRows * kHistRows, kMaxBlocks);
  size_t off = kHeaderBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.hist_cnt = take(sizeof(uint32_t) * kMaxScatter * kMaxBins);
  L.hist_w = take(sizeof(uint64_t) * kMaxBins);
  L.block_hist = take(sizeof(uint32_t) * kMaxBins * blocks);
  L.block_histw = take(sizeof(uint64_t) * kMaxBins * blocks);
  L.block_ranges = take(sizeof(uint32_t) * 4 * blocks);
  L.chunk_part = take(sizeof(uint32_t) * kMaxChunks * kMaxBins);
  L.sub_start = take(sizeof(uint32_t) * kMaxChunks * kMaxBins);
  L.msync = take(sizeof(MidSync));
  L.keys0 = take(8 * (size_t)n);
  L.keys1 = take(8 * (size_t)n);
  L.ids0 = take(4 * (size_t)n);
  L.ids1 = take(4 * (size_t)n);
  L.total = off;
  return L;
}

int d0_bits() {
  const char* e = std::getenv("SEMSCHED_D0");
  const int d = e ? std::atoi(e) : 10;
  return std::min(10, std::max(8, d));
}

// SEMSCHED_FORCE_WIDE=1 makes the global path keep ids in their own array
// even when key and id would share one u64 (the layout very wide key ranges
// need); it lets that layout be exercised on small queues.
int force_wide() {
  const char* e = std::getenv("SEMSCHED_FORCE_WIDE");
  return (e && e[0] == '1') ? 1 : 0;
}

// SEMSCHED_NO_COMPACT=1 keeps the two-pass queues on the u64 element layout
// (the one queues longer than 2^30 requests use), so that layout stays testable.
int no_compact() {
  const char* e = std::getenv("SEMSCHED_NO_COMPACT");
  return (e && e[0] == '1') ? 1 : 0;
}

// SEMSCHED_SPLIT_MID=1 runs the middle passes as separate launches per phase
// (the form a blocking call falls back to when the grid barrier gives up).
int split_mid_forced() {
  const char* e = std::getenv("SEMSCHED_SPLIT_MID");
  return (e && e[0] == '1') ? 1 : 0;
}

int num_cus() {
  static int v = [] {
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
      return prop.multiProcessorCount;
    return 256;
  }();
  return v;
}

int map_flags(uint32_t f) {
  if (f & kFlagDevice) return SEM_EDEVICE;
  if (f & kFlagInval) return SEM_EINVAL;
  if (f & kFlagRange) return SEM_ERANGE;
  return SEM_OK;
}

#define HIP_TRY(expr)                           \
  do {                                          \
    if ((expr) != hipSuccess) return SEM_EDEVICE; \
  } while (0)

// Library state for the blocking calls: one cached workspace per device.
struct State {
  std::mutex mu;
  hipStream_t stream = nullptr;
  std::map<int, std::pair<void*, size_t>> ws;
};
State& state() {
  static State* s = new State();  // never destroyed: the HIP runtime may be gone at exit
  return *s;
}

int cached_workspace(size_t bytes, void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  auto& slot = state().ws[dev];
  if (slot.second < bytes) {
    if (slot.first) {
      HIP_TRY(hipDeviceSynchronize());
      HIP_TRY(hipFree(slot.first));
      slot.first = nullptr;
      slot.second = 0;
    }
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return SEM_ENOMEM;
    slot.first = p;
    slot.second = bytes;
  }
  *out = slot.first;
  return SEM_OK;
}

// One-shot measurement events, armed by sem_trace_stage.
std::mutex& trace_mu() {
  static std::mutex* m = new std::mutex();
  return *m;
}
StageEvents& trace_slots() {
  static StageEvents* e = new StageEvents();
  return *e;
}

int finish(void* ws, hipStream_t st, uint32_t* raw = nullptr) {
  HIP_TRY(hipStreamSynchronize(st));
  uint32_t f = 0;
  HIP_TRY(hipMemcpy(&f, ws, sizeof(f), hipMemcpyDeviceToHost));
  if (raw) *raw = f;
  return map_flags(f);
}

// Set while a blocking call runs a schedule again with the middle passes as
// separate launches per phase (see run_blocking).
thread_local bool t_split_mid = false;

// Polls of the middle-pass grid barrier before it gives up (SEMSCHED_MID_SPIN
// overrides the default, e.g. to test the path that follows).
uint32_t mid_spin_limit() {
  const char* e = std::getenv("SEMSCHED_MID_SPIN");
  return e ? (uint32_t)std::strtoul(e, nullptr, 10) : (1u << 20);
}

// A blocking call: enqueue, synchronise, map the device's flags. When the
// middle passes' grid barrier gave up (its workgroups were not all resident
// on the device), the schedule is run once more with those passes as
// separate launches, which need no residency.
template <typename F>
int run_blocking(void* ws, hipStream_t st, F enqueue) {
  int rc = enqueue();
  if (rc != SEM_OK) return rc;
  uint32_t f = 0;
  rc = finish(ws, st, &f);
  if (rc == SEM_EDEVICE && (f & kFlagDevice)) {
    t_split_mid = true;
    rc = enqueue();
    if (rc == SEM_OK) rc = finish(ws, st);
    t_split_mid = false;
  }
  return rc;
}

// Enqueue one queue (any n >= 0). Arguments already checked.
// payload / pay_pmax (optional, SJF): ranks carried through the long-queue
// path and their largest value; see GArgs. wide_keys: the caller expects key
// ranges that need middle passes.
int enqueue_queue(const uint8_t* p, const int32_t* l, int64_t n, int32_t num_classes,
                  int32_t* order, int64_t* wait, sem_i128* totals, void* ws, hipStream_t st,
                  const uint8_t* payload = nullptr, const uint32_t* pay_pmax = nullptr,
                  bool wide_keys = false) {
  char* base = static_cast<char*>(ws);
  uint32_t* flags = reinterpret_cast<uint32_t*>(base);
  uint64_t* tot = reinterpret_cast<uint64_t*>(totals);
  if (n == 0) {
    if (launch_fill_zero(flags, 1, st) != hipSuccess) return SEM_EDEVICE;
    if (launch_fill_zero(reinterpret_cast<uint32_t*>(tot), 4 * (size_t)(1 + num_classes), st) !=
        hipSuccess)
      return SEM_EDEVICE;
    return SEM_OK;
  }
  if (!needs_global(n)) {
    if (launch_fill_zero(flags, 1, st) != hipSuccess) return SEM_EDEVICE;
    BArgs a = {};
    a.priority = p;
    a.length = l;
    a.offsets = nullptr;
    a.num_segments = 1;
    a.n_single = n;
    a.num_classes = num_classes;
    a.order = order;
    a.wait = wait;
    a.totals = tot;
    a.flags = flags;
    return launch_single_lds(a, st) == hipSuccess ? SEM_OK : SEM_EDEVICE;
  }
  const Layout L = layout_for(n);
  GArgs g = {};
  g.priority = p;
  g.length = l;
  g.n = n;
  g.order = order;
  g.wait = wait;
  g.totals = tot;
  g.num_classes = num_classes;
  g.d0 = d0_bits();
  g.tiles = (int32_t)L.tiles;
  g.force_wide = force_wide();
  g.main = global_first_split(n);
  g.fin = global_final_split(n);
  g.mid = global_mid_split(n);
  // Keys known to be wide take the middle passes as separate launches
  // (faster than the one-launch form, whose scatter phase spills registers;
  // a queue that needs no middle pass then pays for 9 launches that return
  // at once instead of 1).
  g.split_mid = (wide_keys || t_split_mid || split_mid_forced()) ? 1 : 0;
  g.mid_spin = mid_spin_limit();
  g.kchunks = (int32_t)((n + (1ll << kChunkBits) - 1) >> kChunkBits);
  g.kpb = 0;
  while ((1 << g.kpb) < g.kchunks) ++g.kpb;
  // every chunk boundary must fall inside one block of the first pass
  const int64_t block_items = (int64_t)g.main.tpb * kGlobalTile;
  g.chunked = (!no_compact() && g.kchunks <= kMaxChunks &&
               block_items <= (1ll << kChunkBits)) ? 1 : 0;
  g.flags = reinterpret_cast<uint32_t*>(base + L.flags);
  g.sink = reinterpret_cast<uint64_t*>(base + L.sink);
  g.block_ranges = reinterpret_cast<uint32_t*>(base + L.block_ranges);
  g.plan = reinterpret_cast<Plan*>(base + L.plan);
  g.hist_cnt = reinterpret_cast<uint32_t*>(base + L.hist_cnt);
  g.hist_w = reinterpret_cast<uint64_t*>(base + L.hist_w);
  g.block_hist = reinterpret_cast<uint32_t*>(base + L.block_hist);
  g.block_histw = reinterpret_cast<uint64_t*>(base + L.block_histw);
  g.keys[0] = reinterpret_cast<uint64_t*>(base + L.keys0);
  g.keys[1] = reinterpret_cast<uint64_t*>(base + L.keys1);
  g.ids[0] = reinterpret_cast<uint32_t*>(base + L.ids0);
  g.ids[1] = reinterpret_cast<uint32_t*>(base + L.ids1);
  g.chunk_part = reinterpret_cast<uint32_t*>(base + L.chunk_part);
  g.sub_start = reinterpret_cast<uint32_t*>(base + L.sub_start);
  g.msync = reinterpret_cast<MidSync*>(base + L.msync);
  g.payload = payload;
  g.pay_pmax = pay_pmax;
  StageEvents ev = {};
  bool armed = false;
  {
    std::lock_guard<std::mutex> guard(trace_mu());
    for (int k : {SEM_STAGE_HIST, SEM_STAGE_FIRST, SEM_STAGE_FINAL, SEM_STAGE_MID}) {
      ev.before[k] = trace_slots().before[k];
      ev.after[k] = trace_slots().after[k];
      armed = armed || ev.before[k] || ev.after[k];
      trace_slots().before[k] = trace_slots().after[k] = nullptr;
    }
  }
  return launch_global_schedule(g, st, armed ? &ev : nullptr) == hipSuccess ? SEM_OK
                                                                           : SEM_EDEVICE;
}

// Workspace of an insertion: the arrivals' own schedule (its workspace first,
// so that the error flags sit at offset 0), then their order and waits, the
// insertion points, class starts, length totals and scratch totals.
struct InsLayout {
  size_t order_m = 0, wait_m = 0, ins = 0, desc = 0, cs = 0, lsum = 0, sink = 0, totals_m = 0,
         total = 0;
};

InsLayout insert_layout(int64_t n_old, int64_t m) {
  InsLayout L;
  size_t off = align_up(layout_for(m).total);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t m1 = (size_t)std::max<int64_t>(m, 1);  // the merge pass reads entry 0 even if m = 0
  L.order_m = take(4 * m1);
  L.wait_m = take(8 * m1);
  L.ins = take(4 * m1);
  L.desc = take(8 * (size_t)(insert_units(n_old) + 1));
  L.cs = take(4 * 257);
  L.lsum = take(16);
  L.sink = take(16);
  L.totals_m = take(sizeof(sem_i128) * (1 + SEM_MAX_CLASSES));
  L.total = off;
  return L;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return abytes > 0 && bbytes > 0 && x < y + bbytes && y < x + abytes;
}

int check_insert_args(const uint8_t* p, const int32_t* l, int64_t n_old, int64_t m,
                      const int32_t* order_old, const int64_t* wait_old, int32_t* order,
                      int64_t* wait, sem_i128* totals) {
  if (n_old < 0 || m < 0 || n_old + m > INT32_MAX || !totals) return SEM_EINVAL;
  const int64_t n = n_old + m;
  if (n > 0 && (!p || !l || !order || !wait)) return SEM_EINVAL;
  if (n_old > 0 && (!order_old || !wait_old)) return SEM_EINVAL;
  if (overlaps(order, 4 * (size_t)n, order_old, 4 * (size_t)n_old) ||
      overlaps(wait, 8 * (size_t)n, wait_old, 8 * (size_t)n_old) ||
      overlaps(order, 4 * (size_t)n, wait_old, 8 * (size_t)n_old) ||
      overlaps(wait, 8 * (size_t)n, order_old, 4 * (size_t)n_old))
    return SEM_EINVAL;
  return SEM_OK;
}

int enqueue_insert(const uint8_t* p, const int32_t* l, int64_t n_old, int64_t m,
                   const int32_t* order_old, const int64_t* wait_old, int32_t* order,
                   int64_t* wait, sem_i128* totals, void* ws, hipStream_t st) {
  char* base = static_cast<char*>(ws);
  const InsLayout L = insert_layout(n_old, m);
  InsArgs a = {};
  a.priority = p;
  a.length = l;
  a.n_old = n_old;
  a.m = m;
  a.order_old = order_old;
  a.wait_old = wait_old;
  a.order_m = reinterpret_cast<int32_t*>(base + L.order_m);
  a.wait_m = reinterpret_cast<int64_t*>(base + L.wait_m);
  a.ins = reinterpret_cast<uint32_t*>(base + L.ins);
  a.desc = reinterpret_cast<uint64_t*>(base + L.desc);
  a.cs = reinterpret_cast<uint32_t*>(base + L.cs);
  a.lsum = reinterpret_cast<uint64_t*>(base + L.lsum);
  a.sink = reinterpret_cast<uint64_t*>(base + L.sink);
  a.order = order;
  a.wait = wait;
  a.totals = reinterpret_cast<uint64_t*>(totals);
  // the arrivals' own schedule (validates them; resets the error flags)
  int rc = enqueue_queue(p + n_old, l + n_old, m, SEM_MAX_CLASSES,
                         const_cast<int32_t*>(a.order_m), const_cast<int64_t*>(a.wait_m),
                         reinterpret_cast<sem_i128*>(base + L.totals_m), ws, st);
  if (rc != SEM_OK) return rc;
  if (launch_fill_zero(reinterpret_cast<uint32_t*>(totals), 4 * (size_t)(1 + SEM_MAX_CLASSES),
                       st) != hipSuccess)
    return SEM_EDEVICE;
  hipEvent_t before = nullptr, after = nullptr;
  {
    std::lock_guard<std::mutex> guard(trace_mu());
    before = trace_slots().before[SEM_STAGE_MERGE];
    after = trace_slots().after[SEM_STAGE_MERGE];
    trace_slots().before[SEM_STAGE_MERGE] = trace_slots().after[SEM_STAGE_MERGE] = nullptr;
  }
  return launch_insert(a, st, before, after) == hipSuccess ? SEM_OK : SEM_EDEVICE;
}

// Workspace of a comparison-policy schedule. SJF runs the queue kernels on a
// zeroed rank array first, so its layout starts with the queue workspace
// (error flags at offset 0) and that array; FCFS and HPJF use the header's
// flag word. Then the policy kernels' tables.
struct PolLayout {
  size_t zeros = 0, pmax = 0, rsum = 0, tab_cnt = 0, tab_len = 0, ctot_cnt = 0, ctot_len = 0,
         part = 0, sink = 0, total = 0;
};

PolLayout policy_layout(int policy, int64_t n) {
  PolLayout L;
  size_t off = policy == SEM_POLICY_SJF ? align_up(layout_for(n).total) : kHeaderBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t ranges = (size_t)std::max<int64_t>(policy_ranges(n), 1);
  const size_t blocks = (size_t)std::max<int64_t>(policy_blocks(n), 1);
  if (policy == SEM_POLICY_SJF) L.zeros = take(((size_t)n + 3) / 4 * 4);
  L.pmax = take(4);
  if (policy == SEM_POLICY_FCFS) L.rsum = take(8 * ranges);
  if (policy == SEM_POLICY_HPJF) {
    L.tab_cnt = take(4 * ranges * SEM_MAX_CLASSES);
    L.tab_len = take(8 * ranges * SEM_MAX_CLASSES);
    L.ctot_cnt = take(4 * SEM_MAX_CLASSES);
    L.ctot_len = take(8 * SEM_MAX_CLASSES);
  }
  L.part = take(16 * blocks * SEM_MAX_CLASSES);
  L.sink = take(16);
  L.total = off;
  return L;
}

bool known_policy(int policy) {
  return policy == SEM_POLICY_SEMANTIC || policy == SEM_POLICY_FCFS ||
         policy == SEM_POLICY_SJF || policy == SEM_POLICY_HPJF;
}

int check_queue_args(const uint8_t* p, const int32_t* l, int64_t n, int32_t* order,
                     int64_t* wait, sem_i128* totals);

// Workspace of a cost-model schedule: the queue workspace (error flags at
// offset 0), the cost pass's own error word, the service times.
struct CostLayout {
  size_t cflags = 0, service = 0, total = 0;
};

CostLayout cost_layout(int64_t n) {
  CostLayout L;
  size_t off = align_up(layout_for(n).total);
  L.cflags = off;
  off = align_up(off + 4);
  L.service = off;
  off = align_up(off + 4 * (size_t)std::max<int64_t>(n, 1));
  L.total = off;
  return L;
}

CostArgs cost_args(const int32_t* prompt, const int32_t* output, const int32_t* decoded,
                   int64_t n, const sem_cost_model* m) {
  CostArgs a = {};
  a.prompt = prompt;
  a.output = output;
  a.decoded = decoded;
  a.n = n;
  a.alpha1 = m->alpha1;
  a.alpha2 = m->alpha2;
  a.beta = m->beta;
  a.gamma1 = m->gamma1;
  a.gamma2 = m->gamma2;
  return a;
}

int check_cost_args(const int32_t* prompt, const int32_t* output, int64_t n,
                    const sem_cost_model* model, const void* out) {
  if (n < 0 || n > INT32_MAX || !model) return SEM_EINVAL;
  if (n > 0 && (!prompt || !output || !out)) return SEM_EINVAL;
  return SEM_OK;
}

int enqueue_cost_schedule(const uint8_t* p, const int32_t* prompt, const int32_t* output,
                          const int32_t* decoded, int64_t n, const sem_cost_model* model,
                          int32_t* order, int64_t* wait, sem_i128* totals, int32_t* service,
                          void* ws, hipStream_t st) {
  char* base = static_cast<char*>(ws);
  const CostLayout L = cost_layout(n);
  uint32_t* cflags = reinterpret_cast<uint32_t*>(base + L.cflags);
  CostArgs a = cost_args(prompt, output, decoded, n, model);
  a.service = service ? service : reinterpret_cast<int32_t*>(base + L.service);
  a.flags = cflags;
  if (launch_fill_zero(cflags, 1, st) != hipSuccess) return SEM_EDEVICE;
  hipEvent_t before = nullptr, after = nullptr;
  {
    std::lock_guard<std::mutex> guard(trace_mu());
    before = trace_slots().before[SEM_STAGE_COST];
    after = trace_slots().after[SEM_STAGE_COST];
    trace_slots().before[SEM_STAGE_COST] = trace_slots().after[SEM_STAGE_COST] = nullptr;
  }
  if (launch_service(a, st, before, after) != hipSuccess) return SEM_EDEVICE;
  // service times span about 30 bits: two or more middle passes
  const int rc = enqueue_queue(p, a.service, n, SEM_MAX_CLASSES, order, wait, totals, ws, st,
                               nullptr, nullptr, true);
  if (rc != SEM_OK) return rc;
  return launch_merge_flags(reinterpret_cast<uint32_t*>(base), cflags, st) == hipSuccess
             ? SEM_OK
             : SEM_EDEVICE;
}

int enqueue_policy(int policy, const uint8_t* p, const int32_t* l, int64_t n, int32_t* order,
                   int64_t* wait, sem_i128* totals, void* ws, hipStream_t st) {
  if (policy == SEM_POLICY_SEMANTIC)
    return enqueue_queue(p, l, n, SEM_MAX_CLASSES, order, wait, totals, ws, st);
  char* base = static_cast<char*>(ws);
  uint32_t* flags = reinterpret_cast<uint32_t*>(base);
  uint32_t* tot32 = reinterpret_cast<uint32_t*>(totals);
  const size_t tot_words = 4 * (size_t)(1 + SEM_MAX_CLASSES);
  if (n == 0) {
    if (launch_fill_zero(flags, 1, st) != hipSuccess ||
        launch_fill_zero(tot32, tot_words, st) != hipSuccess)
      return SEM_EDEVICE;
    return SEM_OK;
  }
  const PolLayout L = policy_layout(policy, n);
  PolArgs a = {};
  a.priority = p;
  a.length = l;
  a.n = n;
  a.order = order;
  a.wait = wait;
  a.totals = reinterpret_cast<uint64_t*>(totals);
  a.flags = flags;
  a.pmax = reinterpret_cast<uint32_t*>(base + L.pmax);
  a.rsum = reinterpret_cast<uint64_t*>(base + L.rsum);
  a.tab_cnt = reinterpret_cast<uint32_t*>(base + L.tab_cnt);
  a.tab_len = reinterpret_cast<uint64_t*>(base + L.tab_len);
  a.ctot_cnt = reinterpret_cast<uint32_t*>(base + L.ctot_cnt);
  a.ctot_len = reinterpret_cast<uint64_t*>(base + L.ctot_len);
  a.part = reinterpret_cast<uint64_t*>(base + L.part);
  a.sink = reinterpret_cast<uint64_t*>(base + L.sink);
  if (policy == SEM_POLICY_SJF) {
    // The order by (length, id): the queue kernels with every rank read as
    // 0. The largest rank comes first, so that a long queue's compact
    // elements can carry the ranks to its final pass (then that pass splits
    // the totals; else s_classes does, after it).
    uint32_t* zeros = reinterpret_cast<uint32_t*>(base + L.zeros);
    if (launch_fill_zero(zeros, ((size_t)n + 3) / 4, st) != hipSuccess ||
        launch_fill_zero(a.pmax, 1, st) != hipSuccess ||
        launch_policy_range(a, st) != hipSuccess)
      return SEM_EDEVICE;
    const int rc = enqueue_queue(reinterpret_cast<const uint8_t*>(zeros), l, n, SEM_MAX_CLASSES,
                                 order, wait, totals, ws, st, p, a.pmax);
    if (rc != SEM_OK) return rc;
    if (needs_global(n)) a.pay = &reinterpret_cast<const Plan*>(base + layout_for(n).plan)->pay;
  } else if (launch_fill_zero(flags, 1, st) != hipSuccess ||
             launch_fill_zero(a.pmax, 1, st) != hipSuccess ||
             launch_fill_zero(tot32, tot_words, st) != hipSuccess) {
    return SEM_EDEVICE;
  }
  hipEvent_t before = nullptr, after = nullptr;
  {
    std::lock_guard<std::mutex> guard(trace_mu());
    before = trace_slots().before[SEM_STAGE_POLICY];
    after = trace_slots().after[SEM_STAGE_POLICY];
    trace_slots().before[SEM_STAGE_POLICY] = trace_slots().after[SEM_STAGE_POLICY] = nullptr;
  }
  hipError_t e = policy == SEM_POLICY_FCFS   ? launch_fcfs(a, st, before, after)
                 : policy == SEM_POLICY_HPJF ? launch_hpjf(a, st, before, after)
                                             : launch_class_totals(a, st, before, after);
  return e == hipSuccess ? SEM_OK : SEM_EDEVICE;
}

int check_queue_args(const uint8_t* p, const int32_t* l, int64_t n, int32_t* order,
                     int64_t* wait, sem_i128* totals) {
  if (n < 0 || n > INT32_MAX) return SEM_EINVAL;
  if (!totals) return SEM_EINVAL;
  if (n > 0 && (!p || !l || !order || !wait)) return SEM_EINVAL;
  return SEM_OK;
}

int check_batched_args(const uint8_t* p, const int32_t* l, const int64_t* offsets,
                       int64_t num_segments, int32_t num_classes, int32_t* order,
                       int64_t* wait, sem_i128* totals) {
  if (num_segments < 0 || num_segments > INT32_MAX || num_classes < 1 ||
      num_classes > SEM_MAX_CLASSES)
    return SEM_EINVAL;
  if (!offsets) return SEM_EINVAL;
  if (num_segments > 0 && (!p || !l || !order || !wait || !totals)) return SEM_EINVAL;
  return SEM_OK;
}

// Workspace of a batched call: the flags line, the control block, the work
// lists, then the segmented sort's arrays for up to `long_cap` requests in
// queues longer than kSegLargeCap.
struct BLayout {
  size_t ctl = 64, grab = 0, lists = 0, keys0 = 0, keys1 = 0, ids0 = 0, ids1 = 0, hist = 0, tsum = 0,
         lbase = 0, tstart = 0, istart = 0, qtot = 0, tdesc = 0, imap = 0, total = 0;
  uint32_t max_tiles = 0;
};

static_assert(64 + sizeof(BCtl) <= kHeaderBytes, "control block must fit in the header");

BLayout batched_layout(int64_t S, uint64_t long_cap) {
  BLayout L;
  size_t off = kHeaderBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.grab = take(sizeof(GrabLine) * kLists * kSubLists);
  // the medium and wide lists' segments, then the long list
  L.lists = take(4 * (2 * kSubLists * (size_t)list_segment_cap(S) + (size_t)S));
  if (long_cap > 0) {
    const uint64_t queues = std::min<uint64_t>((uint64_t)S, long_cap / (kSegLargeCap + 1));
    L.max_tiles = long_max_tiles(long_cap, S);
    L.keys0 = take(8 * long_cap);
    L.keys1 = take(8 * long_cap);
    L.ids0 = take(4 * long_cap);
    L.ids1 = take(4 * long_cap);
    L.hist = take(4 * ((size_t)1 << kLongDigitBits) * (size_t)L.max_tiles);
    L.tsum = take(8 * (size_t)L.max_tiles);
    L.lbase = take(8 * (size_t)(queues + 1));
    L.tstart = take(4 * (size_t)(queues + 1));
    L.istart = take(4 * (size_t)(queues + 1));
    L.qtot = take(4 * (size_t)kLongColDigits * (size_t)long_items_max(long_cap, (int64_t)queues));
    L.tdesc = take(sizeof(LongTileDesc) * (size_t)L.max_tiles);
    L.imap = take(4 * (size_t)long_items_max(long_cap, (int64_t)queues));
  }
  L.total = off;
  return L;
}

// Largest long-queue capacity whose batched layout fits ws_bytes (0 if only
// the fixed part does).
uint64_t long_capacity(int64_t S, size_t ws_bytes) {
  if (batched_layout(S, 1).total > ws_bytes) return 0;
  uint64_t lo = 1, hi = ws_bytes / 24 + 1;  // more than 24 bytes per request
  while (hi - lo > 1) {
    const uint64_t mid = lo + (hi - lo) / 2;
    if (batched_layout(S, mid).total <= ws_bytes) lo = mid;
    else hi = mid;
  }
  return lo;
}

int enqueue_batched(const uint8_t* p, const int32_t* l, const int64_t* offsets,
                    int64_t num_segments, int32_t num_classes, int32_t* order, int64_t* wait,
                    sem_i128* totals, void* ws, size_t ws_bytes, hipStream_t st) {
  char* base = static_cast<char*>(ws);
  uint32_t* flags = reinterpret_cast<uint32_t*>(base);
  const uint64_t cap = long_capacity(num_segments, ws_bytes);
  const BLayout L = batched_layout(num_segments, cap);
  // the flags line, the control block and the grab counters: one fill
  if (launch_fill_zero(flags, (L.grab + sizeof(GrabLine) * kLists * kSubLists) / 4, st) !=
      hipSuccess)
    return SEM_EDEVICE;
  if (num_segments == 0) return SEM_OK;
  BArgs a = {};
  a.priority = p;
  a.length = l;
  a.offsets = offsets;
  a.num_segments = num_segments;
  a.num_classes = num_classes;
  a.order = order;
  a.wait = wait;
  a.totals = reinterpret_cast<uint64_t*>(totals);
  a.flags = flags;
  a.ctl = reinterpret_cast<BCtl*>(base + L.ctl);
  a.grab = reinterpret_cast<GrabLine*>(base + L.grab);
  a.lists = reinterpret_cast<uint32_t*>(base + L.lists);
  a.seg_cap = list_segment_cap(num_segments);
  a.long_cap = cap;
  a.max_tiles = L.max_tiles;
  if (cap > 0) {
    a.keys[0] = reinterpret_cast<uint64_t*>(base + L.keys0);
    a.keys[1] = reinterpret_cast<uint64_t*>(base + L.keys1);
    a.ids[0] = reinterpret_cast<uint32_t*>(base + L.ids0);
    a.ids[1] = reinterpret_cast<uint32_t*>(base + L.ids1);
    a.hist = reinterpret_cast<uint32_t*>(base + L.hist);
    a.tsum = reinterpret_cast<uint64_t*>(base + L.tsum);
    a.lbase = reinterpret_cast<uint64_t*>(base + L.lbase);
    a.tstart = reinterpret_cast<uint32_t*>(base + L.tstart);
    a.istart = reinterpret_cast<uint32_t*>(base + L.istart);
    a.qtot = reinterpret_cast<uint32_t*>(base + L.qtot);
    a.tdesc = reinterpret_cast<LongTileDesc*>(base + L.tdesc);
    a.imap = reinterpret_cast<uint32_t*>(base + L.imap);
  }
  return launch_batched(a, st) == hipSuccess ? SEM_OK : SEM_EDEVICE;
}

// ---- allocation-free single-queue schedule ---------------------------------
// `scratch` stands in for the workspace of sem_schedule_async when the caller
// cannot allocate one. Every device the library runs on holds its own copy
// until the process ends. In host code the array's name is not a device
// address: each device's address is taken once with hipGetSymbolAddress and
// only that address is handed to kernels.
static __device__ __align__(256) uint8_t scratch[SEM_STATIC_SCRATCH_BYTES];

// Device-side status of the call: the error bits of the flags word mapped to
// the library's codes, written to the caller's status word.
__global__ void g_write_status(const uint32_t* flags, int32_t* status) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    const uint32_t f = *flags;
    *status = (f & kFlagDevice)  ? SEM_EDEVICE
              : (f & kFlagInval) ? SEM_EINVAL
              : (f & kFlagRange) ? SEM_ERANGE
                                 : SEM_OK;
  }
}

// This device's address of `scratch`, looked up once per device.
int scratch_address(void** out) {
  static std::mutex mu;
  static std::map<int, void*> addr;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> guard(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SEM_EDEVICE;
    it = addr.emplace(dev, p).first;
  }
  *out = it->second;
  return SEM_OK;
}

}  // namespace

extern "C" {

int sem_schedule_static(const uint8_t* priority, const int32_t* length, int64_t n,
                        int32_t* order_out, int64_t* wait_out, sem_i128* totals_out,
                        int32_t* status_out, void* stream) {
  int rc = check_queue_args(priority, length, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!status_out) return SEM_EINVAL;
  if (n > SEM_STATIC_MAX_N) return SEM_ENOMEM;
  if (sem_workspace_bytes(n, 1) > SEM_STATIC_SCRATCH_BYTES) return SEM_ENOMEM;
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  rc = enqueue_queue(priority, length, n, SEM_MAX_CLASSES, order_out, wait_out, totals_out, ws,
                     st);
  if (rc != SEM_OK) return rc;
  hipLaunchKernelGGL(g_write_status, dim3(1), dim3(64), 0, st,
                     static_cast<const uint32_t*>(ws), status_out);
  return hipGetLastError() == hipSuccess ? SEM_OK : SEM_EDEVICE;
}

const char* sem_strerror(int code) {
  switch (code) {
    case SEM_OK: return "success";
    case SEM_EINVAL: return "invalid argument";
    case SEM_ERANGE: return "length < 0 or priority >= num_classes";
    case SEM_ENOMEM: return "out of device memory";
    case SEM_EDEVICE: return "HIP runtime error";
    case SEM_ENOTIMPL: return "size beyond what this entry point implements";
    default: return "unknown error";
  }
}

int sem_trace_stage(int stage, void* before, void* after) {
  if (stage < SEM_STAGE_HIST || stage > SEM_STAGE_MID) return SEM_EINVAL;
  std::lock_guard<std::mutex> guard(trace_mu());
  trace_slots().before[stage] = static_cast<hipEvent_t>(before);
  trace_slots().after[stage] = static_cast<hipEvent_t>(after);
  return SEM_OK;
}

int sem_set_stream(void* stream) {
  std::lock_guard<std::mutex> g(state().mu);
  state().stream = static_cast<hipStream_t>(stream);
  return SEM_OK;
}

size_t sem_workspace_bytes(int64_t n, int64_t num_segments) {
  if (n < 0 || num_segments < 0 || num_segments > INT32_MAX) return 0;
  const size_t batched = batched_layout(num_segments, (uint64_t)n).total;
  if (num_segments == 1) return std::max(layout_for(n).total, batched);
  return batched;
}

int sem_check(const void* workspace, void* stream) {
  if (!workspace) return SEM_EINVAL;
  return finish(const_cast<void*>(workspace), static_cast<hipStream_t>(stream));
}

int sem_schedule_async(const uint8_t* priority, const int32_t* length, int64_t n,
                       int32_t* order_out, int64_t* wait_out, sem_i128* totals_out,
                       void* workspace, size_t ws_bytes, void* stream) {
  const int rc = check_queue_args(priority, length, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_workspace_bytes(n, 1) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_queue(priority, length, n, SEM_MAX_CLASSES, order_out, wait_out, totals_out,
                       workspace, static_cast<hipStream_t>(stream));
}

size_t sem_insert_workspace_bytes(int64_t n_old, int64_t m) {
  if (n_old < 0 || m < 0) return 0;
  return insert_layout(n_old, m).total;
}

int sem_insert_async(const uint8_t* priority, const int32_t* length, int64_t n_old, int64_t m,
                     const int32_t* order_old, const int64_t* wait_old, int32_t* order_out,
                     int64_t* wait_out, sem_i128* totals_out, void* workspace, size_t ws_bytes,
                     void* stream) {
  const int rc = check_insert_args(priority, length, n_old, m, order_old, wait_old, order_out,
                                   wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_insert_workspace_bytes(n_old, m) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_insert(priority, length, n_old, m, order_old, wait_old, order_out, wait_out,
                        totals_out, workspace, static_cast<hipStream_t>(stream));
}

int sem_insert(const uint8_t* priority, const int32_t* length, int64_t n_old, int64_t m,
               const int32_t* order_old, const int64_t* wait_old, int32_t* order_out,
               int64_t* wait_out, sem_i128* totals_out) {
  int rc = check_insert_args(priority, length, n_old, m, order_old, wait_old, order_out,
                             wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_insert_workspace_bytes(n_old, m), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  return run_blocking(ws, st, [&] {
    return enqueue_insert(priority, length, n_old, m, order_old, wait_old, order_out, wait_out,
                          totals_out, ws, st);
  });
}

size_t sem_policy_workspace_bytes(int policy, int64_t n) {
  if (n < 0 || !known_policy(policy)) return 0;
  if (policy == SEM_POLICY_SEMANTIC) return sem_workspace_bytes(n, 1);
  return policy_layout(policy, n).total;
}

int sem_schedule_policy_async(int policy, const uint8_t* priority, const int32_t* length,
                              int64_t n, int32_t* order_out, int64_t* wait_out,
                              sem_i128* totals_out, void* workspace, size_t ws_bytes,
                              void* stream) {
  if (!known_policy(policy)) return SEM_EINVAL;
  const int rc = check_queue_args(priority, length, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_policy_workspace_bytes(policy, n) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_policy(policy, priority, length, n, order_out, wait_out, totals_out, workspace,
                        static_cast<hipStream_t>(stream));
}

int sem_schedule_policy(int policy, const uint8_t* priority, const int32_t* length, int64_t n,
                        int32_t* order_out, int64_t* wait_out, sem_i128* totals_out) {
  if (!known_policy(policy)) return SEM_EINVAL;
  int rc = check_queue_args(priority, length, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_policy_workspace_bytes(policy, n), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  return run_blocking(ws, st, [&] {
    return enqueue_policy(policy, priority, length, n, order_out, wait_out, totals_out, ws, st);
  });
}

int sem_service_times(const int32_t* prompt, const int32_t* output, const int32_t* decoded,
                      int64_t n, const sem_cost_model* model, int32_t* service_out) {
  int rc = check_cost_args(prompt, output, n, model, service_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(kHeaderBytes, &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  CostArgs a = cost_args(prompt, output, decoded, n, model);
  a.service = service_out;
  a.flags = static_cast<uint32_t*>(ws);
  if (launch_fill_zero(a.flags, 1, st) != hipSuccess ||
      launch_service(a, st, nullptr, nullptr) != hipSuccess)
    return SEM_EDEVICE;
  return finish(ws, st);
}

int sem_evict_plan(const int32_t* prompt, const int32_t* decoded, int64_t n,
                   const sem_cost_model* model, uint8_t* keep_prefill_out,
                   int32_t* save_tokens_out) {
  int rc = check_cost_args(prompt, decoded, n, model, keep_prefill_out);
  if (rc != SEM_OK) return rc;
  if (n > 0 && !save_tokens_out) return SEM_EINVAL;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(kHeaderBytes, &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  CostArgs a = cost_args(prompt, nullptr, decoded, n, model);
  a.keep = keep_prefill_out;
  a.save = save_tokens_out;
  a.flags = static_cast<uint32_t*>(ws);
  if (launch_fill_zero(a.flags, 1, st) != hipSuccess || launch_evict(a, st) != hipSuccess)
    return SEM_EDEVICE;
  return finish(ws, st);
}

size_t sem_cost_workspace_bytes(int64_t n) {
  if (n < 0) return 0;
  return cost_layout(n).total;
}

int sem_schedule_cost_async(const uint8_t* priority, const int32_t* prompt, const int32_t* output,
                            const int32_t* decoded, int64_t n, const sem_cost_model* model,
                            int32_t* order_out, int64_t* wait_out, sem_i128* totals_out,
                            int32_t* service_out, void* workspace, size_t ws_bytes,
                            void* stream) {
  int rc = check_cost_args(prompt, output, n, model, order_out);
  if (rc != SEM_OK) return rc;
  rc = check_queue_args(priority, prompt, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_cost_workspace_bytes(n) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_cost_schedule(priority, prompt, output, decoded, n, model, order_out, wait_out,
                               totals_out, service_out, workspace,
                               static_cast<hipStream_t>(stream));
}

int sem_schedule_cost(const uint8_t* priority, const int32_t* prompt, const int32_t* output,
                      const int32_t* decoded, int64_t n, const sem_cost_model* model,
                      int32_t* order_out, int64_t* wait_out, sem_i128* totals_out,
                      int32_t* service_out) {
  int rc = check_cost_args(prompt, output, n, model, order_out);
  if (rc != SEM_OK) return rc;
  rc = check_queue_args(priority, prompt, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_cost_workspace_bytes(n), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  return run_blocking(ws, st, [&] {
    return enqueue_cost_schedule(priority, prompt, output, decoded, n, model, order_out, wait_out,
                                 totals_out, service_out, ws, st);
  });
}

static_assert(SEM_SELECT_CAP == kSelectCap && SEM_EVICT_CAP == kEvictCap,
              "the header's LDS sizes are the kernels'");
static_assert(SEM_WIDE_MAX == kWideMax, "the header's largest lists are the kernels'");

// Selection and eviction: one workgroup over LDS up to the SEM_*_CAP sizes;
// beyond them the workspace holds the sort buffers of the lists (two
// ping-pong buffers of keys, ids and, for eviction, indices into the caller's
// arrays), then the kept-member prefix (selection) or the KV prefix sums and
// the eviction order (eviction).
bool select_in_lds(int64_t n_buffer, int64_t n_ongoing, int64_t b) {
  return b <= kSelectCap && n_buffer <= kSelectCap && n_ongoing <= kSelectCap;
}

struct WideLayout {
  size_t key[2] = {0, 0}, id[2] = {0, 0}, pay[2] = {0, 0}, dec = 0, psum = 0, eorder = 0;
  size_t total = kHeaderBytes;
};

static WideLayout wide_layout(int64_t entries, bool evict) {
  WideLayout L;
  size_t off = kHeaderBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t n = (size_t)entries;
  for (int k = 0; k < 2; ++k) L.key[k] = take(8 * n);
  for (int k = 0; k < 2; ++k) L.id[k] = take(4 * n);
  if (evict) {
    for (int k = 0; k < 2; ++k) L.pay[k] = take(4 * n);
    L.psum = take(8 * n);
    L.eorder = take(4 * n);
  } else {
    L.dec = take(4 * (n + 1));
  }
  L.total = off;
  return L;
}

int64_t select_entries(int64_t n_heap, int64_t n_buffer, int64_t n_ongoing, int64_t b) {
  return std::min(b, n_heap) + n_buffer + n_ongoing;
}

size_t sem_select_workspace_bytes(int64_t n_heap, int64_t n_buffer, int64_t n_ongoing,
                                  int64_t b) {
  if (n_heap < 0 || n_buffer < 0 || n_ongoing < 0 || b < 0) return 0;
  if (select_in_lds(n_buffer, n_ongoing, b)) return kHeaderBytes;
  return wide_layout(select_entries(n_heap, n_buffer, n_ongoing, b), false).total;
}

size_t sem_evict_workspace_bytes(int64_t n_cached) {
  if (n_cached < 0) return 0;
  if (n_cached <= kEvictCap) return kHeaderBytes;
  return wide_layout(n_cached, true).total;
}

int check_select(const uint8_t* p, const int32_t* l, const uint8_t* stage, int64_t n_ids,
                 const int32_t* heap, int64_t n_heap, const int32_t* buffer, int64_t n_buffer,
                 const int32_t* ongoing, int64_t n_ongoing, int64_t b, int32_t* batch,
                 int32_t* pushed, int64_t* counts) {
  if (n_ids < 0 || n_ids > INT32_MAX || n_heap < 0 || n_buffer < 0 || n_ongoing < 0 || b < 0)
    return SEM_EINVAL;
  if (select_entries(n_heap, n_buffer, n_ongoing, b) > kWideMax) return SEM_ENOTIMPL;
  if (!counts) return SEM_EINVAL;
  const bool any = std::min(b, n_heap) + n_buffer + n_ongoing > 0;
  if (any && (!p || !l || !stage)) return SEM_EINVAL;
  if ((std::min(b, n_heap) > 0 && !heap) || (n_buffer > 0 && !buffer) ||
      (n_ongoing > 0 && !ongoing) || (b > 0 && !batch) || (any && !pushed))
    return SEM_EINVAL;
  return SEM_OK;
}

int enqueue_select(const uint8_t* p, const int32_t* l, const uint8_t* stage, int64_t n_ids,
                   const int32_t* heap, int64_t n_heap, const int32_t* buffer, int64_t n_buffer,
                   const int32_t* ongoing, int64_t n_ongoing, int64_t b, int32_t* batch,
                   int32_t* pushed, int64_t* counts, void* ws, hipStream_t st) {
  SelArgs a = {p, l, stage, n_ids, heap, n_heap, buffer, n_buffer, ongoing, n_ongoing, b,
               batch, pushed, counts, static_cast<uint32_t*>(ws)};
  if (launch_fill_zero(a.flags, 1, st) != hipSuccess) return SEM_EDEVICE;
  if (select_in_lds(n_buffer, n_ongoing, b))
    return launch_select(a, st) == hipSuccess ? SEM_OK : SEM_EDEVICE;
  // candidates (the heap's first b, then the buffer) and ongoing requests
  const int64_t nh = std::min(b, n_heap);
  const WideLayout L = wide_layout(nh + n_buffer + n_ongoing, false);
  char* base = static_cast<char*>(ws);
  WideSort w = {};
  w.priority = p;
  w.length = l;
  w.n_ids = n_ids;
  w.kv = nullptr;
  w.list[0] = {heap, nh, buffer, n_buffer, 0};
  w.list[1] = {ongoing, n_ongoing, nullptr, 0, nh + n_buffer};
  w.nlists = 2;
  w.total = nh + n_buffer + n_ongoing;
  for (int k = 0; k < 2; ++k) {
    w.key[k] = reinterpret_cast<uint64_t*>(base + L.key[k]);
    w.id[k] = reinterpret_cast<uint32_t*>(base + L.id[k]);
    w.pay[k] = nullptr;
  }
  w.flags = a.flags;
  return launch_select_wide(a, w, reinterpret_cast<uint32_t*>(base + L.dec), st) == hipSuccess
             ? SEM_OK
             : SEM_EDEVICE;
}

int sem_select_batch_async(const uint8_t* priority, const int32_t* length, const uint8_t* stage,
                           int64_t n_ids, const int32_t* heap_order, int64_t n_heap,
                           const int32_t* buffer, int64_t n_buffer, const int32_t* ongoing,
                           int64_t n_ongoing, int64_t b, int32_t* batch_out, int32_t* pushed_out,
                           int64_t* counts_out, void* workspace, size_t ws_bytes, void* stream) {
  const int rc = check_select(priority, length, stage, n_ids, heap_order, n_heap, buffer,
                              n_buffer, ongoing, n_ongoing, b, batch_out, pushed_out, counts_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_select_workspace_bytes(n_heap, n_buffer, n_ongoing, b) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_select(priority, length, stage, n_ids, heap_order, n_heap, buffer, n_buffer,
                        ongoing, n_ongoing, b, batch_out, pushed_out, counts_out, workspace,
                        static_cast<hipStream_t>(stream));
}

int sem_select_batch(const uint8_t* priority, const int32_t* length, const uint8_t* stage,
                     int64_t n_ids, const int32_t* heap_order, int64_t n_heap,
                     const int32_t* buffer, int64_t n_buffer, const int32_t* ongoing,
                     int64_t n_ongoing, int64_t b, int32_t* batch_out, int32_t* pushed_out,
                     int64_t* counts_out) {
  int rc = check_select(priority, length, stage, n_ids, heap_order, n_heap, buffer, n_buffer,
                        ongoing, n_ongoing, b, batch_out, pushed_out, counts_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_select_workspace_bytes(n_heap, n_buffer, n_ongoing, b), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  rc = enqueue_select(priority, length, stage, n_ids, heap_order, n_heap, buffer, n_buffer,
                      ongoing, n_ongoing, b, batch_out, pushed_out, counts_out, ws, st);
  if (rc != SEM_OK) return rc;
  return finish(ws, st);
}

int check_evict(const uint8_t* p, const int32_t* l, int64_t n_ids, const int32_t* cached,
                const int64_t* kv, int64_t n_cached, const int64_t* demands, int64_t n_demands,
                int32_t* victims, int64_t* upto) {
  if (n_ids < 0 || n_ids > INT32_MAX || n_cached < 0 || n_demands < 0) return SEM_EINVAL;
  if (n_cached > kWideMax) return SEM_ENOTIMPL;
  if (n_cached > 0 && (!p || !l || !cached || !kv || !victims)) return SEM_EINVAL;
  if (n_demands > 0 && (!demands || !upto)) return SEM_EINVAL;
  return SEM_OK;
}

int enqueue_evict(const uint8_t* p, const int32_t* l, int64_t n_ids, const int32_t* cached,
                  const int64_t* kv, int64_t n_cached, int64_t usage, int64_t capacity,
                  const int64_t* demands, int64_t n_demands, int32_t* victims, int64_t* upto,
                  void* ws, hipStream_t st) {
  EvictArgs a = {p, l, n_ids, cached, kv, n_cached, usage, capacity, demands, n_demands,
                 victims, upto, static_cast<uint32_t*>(ws)};
  if (launch_fill_zero(a.flags, 1, st) != hipSuccess) return SEM_EDEVICE;
  if (n_cached + n_demands == 0) return SEM_OK;
  if (n_cached <= kEvictCap)
    return launch_evict_victims(a, st) == hipSuccess ? SEM_OK : SEM_EDEVICE;
  const WideLayout L = wide_layout(n_cached, true);
  char* base = static_cast<char*>(ws);
  WideSort w = {};
  w.priority = p;
  w.length = l;
  w.n_ids = n_ids;
  w.kv = kv;
  w.list[0] = {cached, n_cached, nullptr, 0, 0};
  w.list[1] = {nullptr, 0, nullptr, 0, n_cached};
  w.nlists = 1;
  w.total = n_cached;
  for (int k = 0; k < 2; ++k) {
    w.key[k] = reinterpret_cast<uint64_t*>(base + L.key[k]);
    w.id[k] = reinterpret_cast<uint32_t*>(base + L.id[k]);
    w.pay[k] = reinterpret_cast<uint32_t*>(base + L.pay[k]);
  }
  w.flags = a.flags;
  return launch_evict_wide(a, w, reinterpret_cast<uint64_t*>(base + L.psum),
                           reinterpret_cast<uint32_t*>(base + L.eorder), st) == hipSuccess
             ? SEM_OK
             : SEM_EDEVICE;
}

int sem_evict_async(const uint8_t* priority, const int32_t* length, int64_t n_ids,
                    const int32_t* cached, const int64_t* kv, int64_t n_cached, int64_t usage,
                    int64_t capacity, const int64_t* demands, int64_t n_demands,
                    int32_t* victims_out, int64_t* upto_out, void* workspace, size_t ws_bytes,
                    void* stream) {
  const int rc = check_evict(priority, length, n_ids, cached, kv, n_cached, demands, n_demands,
                             victims_out, upto_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < sem_evict_workspace_bytes(n_cached) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_evict(priority, length, n_ids, cached, kv, n_cached, usage, capacity, demands,
                       n_demands, victims_out, upto_out, workspace,
                       static_cast<hipStream_t>(stream));
}

int sem_evict(const uint8_t* priority, const int32_t* length, int64_t n_ids,
              const int32_t* cached, const int64_t* kv, int64_t n_cached, int64_t usage,
              int64_t capacity, const int64_t* demands, int64_t n_demands, int32_t* victims_out,
              int64_t* upto_out) {
  int rc = check_evict(priority, length, n_ids, cached, kv, n_cached, demands, n_demands,
                       victims_out, upto_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_evict_workspace_bytes(n_cached), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  rc = enqueue_evict(priority, length, n_ids, cached, kv, n_cached, usage, capacity, demands,
                     n_demands, victims_out, upto_out, ws, st);
  if (rc != SEM_OK) return rc;
  return finish(ws, st);
}

int sem_schedule(const uint8_t* priority, const int32_t* length, int64_t n, int32_t* order_out,
                 int64_t* wait_out, sem_i128* totals_out) {
  int rc = check_queue_args(priority, length, n, order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  void* ws = nullptr;
  rc = cached_workspace(sem_workspace_bytes(n, 1), &ws);
  if (rc != SEM_OK) return rc;
  const hipStream_t st = state().stream;
  return run_blocking(ws, st, [&] {
    return enqueue_queue(priority, length, n, SEM_MAX_CLASSES, order_out, wait_out, totals_out,
                         ws, st);
  });
}

int sem_schedule_batched_async(const uint8_t* priority, const int32_t* length,
                               const int64_t* offsets, int64_t num_segments,
                               int32_t num_classes, int32_t* order_out, int64_t* wait_out,
                               sem_i128* totals_out, void* workspace, size_t ws_bytes,
                               void* stream) {
  const int rc = check_batched_args(priority, length, offsets, num_segments, num_classes,
                                    order_out, wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  if (!workspace || ws_bytes < batched_layout(num_segments, 0).total ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return SEM_EINVAL;
  return enqueue_batched(priority, length, offsets, num_segments, num_classes, order_out,
                         wait_out, totals_out, workspace, ws_bytes,
                         static_cast<hipStream_t>(stream));
}

int sem_schedule_batched(const uint8_t* priority, const int32_t* length,
                         const int64_t* offsets, int64_t num_segments, int32_t num_classes,
                         int32_t* order_out, int64_t* wait_out, sem_i128* totals_out) {
  int rc = check_batched_args(priority, length, offsets, num_segments, num_classes, order_out,
                              wait_out, totals_out);
  if (rc != SEM_OK) return rc;
  std::lock_guard<std::mutex> g(state().mu);
  const hipStream_t st = state().stream;
  // the offsets are read once, to size the workspace of the long queues
  std::vector<int64_t> off((size_t)num_segments + 1);
  HIP_TRY(hipMemcpyAsync(off.data(), offsets, off.size() * sizeof(int64_t),
                         hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (off[0] != 0) return SEM_EINVAL;
  uint64_t long_elems = 0;
  for (int64_t s = 0; s < num_segments; ++s) {
    const int64_t m = off[s + 1] - off[s];
    if (m < 0 || m > INT32_MAX) return SEM_EINVAL;
    if (m > kSegLargeCap) long_elems += (uint64_t)m;
  }
  const size_t need = batched_layout(num_segments, long_elems).total;
  void* ws = nullptr;
  rc = cached_workspace(need, &ws);
  if (rc != SEM_OK) return rc;
  rc = enqueue_batched(priority, length, offsets, num_segments, num_classes, order_out,
                       wait_out, totals_out, ws, need, st);
  if (rc != SEM_OK) return rc;
  return finish(ws, st);
}

}  // extern "C"
