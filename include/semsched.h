/*
 * semsched.h — C ABI of the MI355X (gfx950) semantic-scheduling hot path.
 *
 * What the library computes (the paper's Section 3.2 problem statement with
 * all arrivals at time 0 and one server, and Section 3.3's priority tuple):
 *
 *   Each request i has an urgency rank priority[i] (Definition 1: the graded
 *   poset's rank, 0 = most urgent ESI level) and a predicted service time
 *   length[i] (the estimated remaining computation time f_t, here the
 *   predicted generation length in tokens).
 *
 *   order  : request ids ascending by (priority, length, id). This is the
 *            sequence obtained by draining the min-heap keyed by (f_e, f_t)
 *            of Algorithm 1 (MinHeap Construction); under Eq. 2 (relative
 *            constraint) it minimises the total waiting time of Eq. 1. Exact
 *            (priority, length) ties go to the lower id (the paper gives no
 *            tie rule; this one makes the schedule unique).
 *   wait   : wait[k] = sum of length[order[j]] for j < k, int64, in schedule
 *            order (wait[k] belongs to request order[k]). It is the time
 *            before service starts; Eq. 1's finish-minus-arrival is
 *            wait[k] + length[order[k]].
 *   totals : totals[0] = sum of all waits; totals[1 + c] = sum of the waits
 *            of class c (zero for an empty class). Exact signed 128-bit.
 *
 * Memory: every array argument is a DEVICE pointer (e.g. a torch ROCm
 * tensor's data_ptr()) on the current HIP device, except where noted. Inputs
 * are read only. Outputs are caller-owned and fully overwritten; after a
 * failed call their contents are unspecified.
 *
 * Streams: `stream` arguments are a hipStream_t passed as void * (NULL = the
 * null stream). The blocking calls run on the stream set by sem_set_stream
 * and synchronise it before returning.
 *
 * Errors (return values):
 *   SEM_OK       success.
 *   SEM_EINVAL   null pointer with n > 0, n < 0 or n > INT32_MAX,
 *                num_classes outside [1, 256], offsets not starting at 0,
 *                decreasing, or not ending at the total, workspace too small.
 *   SEM_ERANGE   some length < 0, or some priority >= num_classes (256 for
 *                the single-queue calls). Detected on the device.
 *   SEM_ENOMEM   the library could not allocate its internal workspace.
 *   SEM_EDEVICE  a HIP runtime call failed, or (asynchronous calls only) the
 *                grid barrier of the middle passes, needed only by very wide
 *                key ranges, gave up waiting because its workgroups were not
 *                all resident on the device (another program holding compute
 *                units); the outputs are then not written, and running the
 *                call again, or its blocking form, is safe. The blocking
 *                calls handle that case themselves by running the schedule
 *                again with the middle passes as separate launches.
 *   SEM_ENOTIMPL a size beyond what an entry point implements (noted at the
 *                entry points that can return it).
 */
#ifndef SEMSCHED_H
#define SEMSCHED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Exact signed 128-bit integer, two's complement, little-endian words:
 * value = hi * 2^64 + lo. Same layout as __int128 on x86-64 and gfx950. */
typedef struct {
  uint64_t lo;
  int64_t hi;
} sem_i128;

#define SEM_MAX_CLASSES 256 /* priority is uint8 */
#define SEM_SEGMENT_CAP 16384 /* longest queue scheduled inside one workgroup's LDS */

enum {
  SEM_OK = 0,
  SEM_EINVAL = -1,
  SEM_ERANGE = -2,
  SEM_ENOMEM = -3,
  SEM_EDEVICE = -4,
  SEM_ENOTIMPL = -5
};

/*
 * Schedule one queue of n requests (blocking).
 *   priority  [n] uint8, rank of each request (0 = most urgent).
 *   length    [n] int32, predicted service time, must be >= 0.
 *   order_out [n] int32, ids in schedule order.
 *   wait_out  [n] int64, wait of the request at each schedule position.
 *   totals_out[1 + 256] sem_i128, total then per-class waits.
 * Uses a workspace cached by the library (allocated on first need, grown as
 * needed, freed at process exit). n = 0 is valid and zeroes totals_out.
 */
int sem_schedule(const uint8_t *priority, const int32_t *length, int64_t n,
                 int32_t *order_out, int64_t *wait_out, sem_i128 *totals_out);

/*
 * Schedule num_segments independent queues laid out back to back (blocking).
 * Each queue is scheduled exactly as sem_schedule schedules a single queue
 * (Section 3.2 per queue; the paper puts no bound on a queue's length).
 *   offsets   [num_segments + 1] int64, DEVICE pointer; queue s holds
 *             requests offsets[s] .. offsets[s+1]-1. Empty queues are valid.
 *             offsets[0] must be 0 and the offsets non-decreasing; the batch
 *             holds N = offsets[num_segments] requests.
 *   num_classes in [1, 256]: every priority must be below it.
 *   order_out [N] int32, ids LOCAL to each queue (0-based arrival index),
 *             queue s's schedule written at offsets[s] + k.
 *   wait_out  [N] int64, same layout; waits restart at 0 in every queue.
 *   totals_out[num_segments * (1 + num_classes)] sem_i128, queue-major:
 *             queue s's total at s*(1+num_classes), class c at +1+c.
 * Queues of any length are accepted. Queues of up to SEM_SEGMENT_CAP
 * requests are scheduled one per wave or workgroup inside LDS, longer ones by
 * one segmented radix sort over all of them. The call copies the offsets to
 * the host once, to size the workspace of the long queues, and synchronises
 * once at the end.
 */
int sem_schedule_batched(const uint8_t *priority, const int32_t *length,
                         const int64_t *offsets, int64_t num_segments,
                         int32_t num_classes, int32_t *order_out,
                         int64_t *wait_out, sem_i128 *totals_out);

/*
 * Workspace size in bytes needed by the asynchronous calls.
 *   sem_schedule_async: n requests, num_segments = 1.
 *   sem_schedule_batched_async: num_segments queues, n = an upper bound on the
 *     number of requests that lie in queues longer than SEM_SEGMENT_CAP (the
 *     total N when unknown, 0 when every queue is known to be short).
 * With num_segments = 1 the larger of the two sizes is returned.
 */
size_t sem_workspace_bytes(int64_t n, int64_t num_segments);

/*
 * Asynchronous single-queue schedule: same arguments as sem_schedule plus a
 * caller-owned DEVICE workspace of at least sem_workspace_bytes(n, 1) bytes
 * (256-byte aligned) and the stream to enqueue on. Allocates nothing and
 * does not synchronise. Host-detectable argument errors are returned at
 * once; device-detected range errors are left in the workspace and returned
 * by sem_check. A workspace must not be shared by calls in flight at the
 * same time.
 */
int sem_schedule_async(const uint8_t *priority, const int32_t *length,
                       int64_t n, int32_t *order_out, int64_t *wait_out,
                       sem_i128 *totals_out, void *workspace, size_t ws_bytes,
                       void *stream);

/*
 * Asynchronous batched schedule: the arguments of sem_schedule_batched plus a
 * caller-owned DEVICE workspace (256-byte aligned) of ws_bytes bytes and the
 * stream. Allocates nothing, does not synchronise and never reads device
 * memory on the host: the offsets are checked, the queues sorted into work
 * lists by size and the long queues sized on the device. The workspace must
 * hold at least sem_workspace_bytes(0, num_segments) bytes (else SEM_EINVAL
 * at once); whatever it holds beyond that is room for the requests of queues
 * longer than SEM_SEGMENT_CAP, and sem_workspace_bytes(L, num_segments) bytes
 * give room for L of them. Device-detected errors, returned by sem_check:
 * SEM_EINVAL for bad offsets or long queues that do not fit the workspace,
 * SEM_ERANGE for a length < 0 or a priority >= num_classes.
 */
int sem_schedule_batched_async(const uint8_t *priority, const int32_t *length,
                               const int64_t *offsets, int64_t num_segments,
                               int32_t num_classes, int32_t *order_out,
                               int64_t *wait_out, sem_i128 *totals_out,
                               void *workspace, size_t ws_bytes, void *stream);

/*
 * Insert m newly arrived requests into an existing schedule (blocking): the
 * data-parallel form of Algorithm 1's HeapInsert under the asynchronous queue
 * management of Section 3.3 (arrivals join the heap that already holds the
 * earlier requests; draining it gives the schedule of all of them).
 *   priority, length [n_old + m] DEVICE: requests 0 .. n_old-1 are the earlier
 *             ones, n_old .. n_old+m-1 the arrivals (ids continue the arrival
 *             index, so an exact (priority, length) tie goes to the earlier
 *             request).
 *   order_old, wait_old [n_old] DEVICE: the schedule of requests 0 .. n_old-1
 *             as sem_schedule returned it (read only).
 *   order_out, wait_out [n_old + m], totals_out [1 + 256] DEVICE: the schedule
 *             of all n_old + m requests, identical to what sem_schedule returns
 *             for them. The outputs must not overlap order_old / wait_old.
 * Only the arrivals are sorted; every earlier entry is read and written once.
 * Errors: SEM_EINVAL (n_old or m < 0, n_old + m > INT32_MAX, null pointers,
 * overlapping outputs), SEM_ERANGE (an arrival's length < 0). If order_old /
 * wait_old are not the schedule of the earlier requests the result is
 * unspecified, but no memory outside the arguments is accessed.
 */
int sem_insert(const uint8_t *priority, const int32_t *length, int64_t n_old,
               int64_t m, const int32_t *order_old, const int64_t *wait_old,
               int32_t *order_out, int64_t *wait_out, sem_i128 *totals_out);

/* Workspace size in bytes needed by sem_insert_async. */
size_t sem_insert_workspace_bytes(int64_t n_old, int64_t m);

/*
 * Asynchronous sem_insert: same arguments plus a caller-owned DEVICE
 * workspace of at least sem_insert_workspace_bytes(n_old, m) bytes (256-byte
 * aligned) and the stream; allocates nothing, does not synchronise; an
 * arrival's range error is returned by sem_check(workspace, stream).
 */
int sem_insert_async(const uint8_t *priority, const int32_t *length,
                     int64_t n_old, int64_t m, const int32_t *order_old,
                     const int64_t *wait_old, int32_t *order_out,
                     int64_t *wait_out, sem_i128 *totals_out, void *workspace,
                     size_t ws_bytes, void *stream);

/*
 * Comparison policies: the baselines of the request-spike experiments of
 * Section 4 (first-come-first-served, shortest job first, highest-priority
 * job first), plus the semantic order itself. Each keys the order by some
 * fields of the request and closes the key with the id:
 *   SEM_POLICY_SEMANTIC  (priority, length, id): the same as sem_schedule
 *   SEM_POLICY_FCFS      (id): arrival order
 *   SEM_POLICY_SJF       (length, id): the rank is ignored
 *   SEM_POLICY_HPJF      (priority, id): the length is ignored
 */
#define SEM_POLICY_SEMANTIC 0
#define SEM_POLICY_FCFS 1
#define SEM_POLICY_SJF 2
#define SEM_POLICY_HPJF 3

/*
 * Schedule one queue under `policy` (blocking). Arguments, layouts and
 * outputs as for sem_schedule: wait_out[k] is the exclusive prefix of the
 * lengths in the policy's order, totals_out[1 + c] the sum of the waits of
 * the requests whose priority is c (whatever the policy orders by).
 * Errors: SEM_EINVAL for an unknown policy, else as sem_schedule (a negative
 * length is SEM_ERANGE under every policy, FCFS included).
 */
int sem_schedule_policy(int policy, const uint8_t *priority, const int32_t *length,
                        int64_t n, int32_t *order_out, int64_t *wait_out,
                        sem_i128 *totals_out);

/* Workspace size in bytes of sem_schedule_policy_async (0 for an unknown
 * policy or n < 0). */
size_t sem_policy_workspace_bytes(int policy, int64_t n);

/* Asynchronous sem_schedule_policy: a caller-owned DEVICE workspace of at
 * least sem_policy_workspace_bytes(policy, n) bytes (256-byte aligned) and
 * the stream; allocates nothing, does not synchronise; range errors are
 * returned by sem_check(workspace, stream). */
int sem_schedule_policy_async(int policy, const uint8_t *priority, const int32_t *length,
                              int64_t n, int32_t *order_out, int64_t *wait_out,
                              sem_i128 *totals_out, void *workspace, size_t ws_bytes,
                              void *stream);

/*
 * Cost model of Section 3.4. Constants are unsigned Q32.32 fixed point: a
 * value v means v / 2^32 time units (the caller's unit, e.g. microseconds)
 * per token (alpha2, beta, gamma1, gamma2) or per token^2 (alpha1):
 *   prefill of n prompt tokens:     alpha1 * n^2 + alpha2 * n
 *   reloading n tokens of KV cache: beta * n
 *   decoding tokens n+1 .. n+m:     gamma1 * (m^2/2 + n*m + m/2) + gamma2 * m  (Eq. 4)
 * Every product and sum is exact (128-bit); results are deterministic integers.
 */
typedef struct {
  uint64_t alpha1, alpha2, beta, gamma1, gamma2;
} sem_cost_model;

/*
 * Remaining computation time of each request (blocking), the f_t of the
 * scheduling tuple: for prompt[i] tokens, output[i] predicted output tokens
 * and decoded[i] tokens decoded so far (decoded may be NULL: all 0), the
 * cost of decoding tokens prompt+decoded+1 .. prompt+output (none once
 * decoded >= output) plus the prefill while decoded = 0, as
 * floor(cost / 2^32) time units, saturated at 2^31 - 1.
 *   prompt, output, decoded [n] int32 DEVICE; model HOST pointer;
 *   service_out [n] int32 DEVICE.
 * Errors: SEM_EINVAL (n < 0 or > INT32_MAX, null pointers), SEM_ERANGE (a
 * negative count; that request's service time is written as 0).
 */
int sem_service_times(const int32_t *prompt, const int32_t *output, const int32_t *decoded,
                      int64_t n, const sem_cost_model *model, int32_t *service_out);

/*
 * Cache decisions for n evicted requests (blocking; Algorithm 4's
 * ShouldRecompute and the decode-stage split of Section 3.4):
 *   keep_prefill_out[i] = 1 when reloading the prompt's cache is cheaper
 *     than recomputing it: beta * p < alpha1 * p^2 + alpha2 * p for
 *     p = prompt[i] (Eq. 3 with the comparison its explanation implies);
 *   save_tokens_out[i] = the number x in [0, decoded[i]] of decoded tokens
 *     whose cache to save that minimises Eq. 5,
 *     beta * x + gamma1 * (y^2/2 + p*y + y/2) + gamma2 * y with y = decoded - x,
 *     the largest such x among equal costs (exact integer minimiser).
 *   prompt, decoded [n] int32 DEVICE; keep_prefill_out [n] uint8 and
 *   save_tokens_out [n] int32 DEVICE. Errors as sem_service_times.
 */
int sem_evict_plan(const int32_t *prompt, const int32_t *decoded, int64_t n,
                   const sem_cost_model *model, uint8_t *keep_prefill_out,
                   int32_t *save_tokens_out);

/*
 * Schedule one queue by (priority, cost-model service time, id) (blocking):
 * sem_service_times followed by sem_schedule on those times. service_out
 * ([n] int32 DEVICE) receives the service times when not NULL. Outputs and
 * errors as sem_schedule and sem_service_times.
 */
int sem_schedule_cost(const uint8_t *priority, const int32_t *prompt, const int32_t *output,
                      const int32_t *decoded, int64_t n, const sem_cost_model *model,
                      int32_t *order_out, int64_t *wait_out, sem_i128 *totals_out,
                      int32_t *service_out);

/* Workspace size in bytes of sem_schedule_cost_async for n requests. */
size_t sem_cost_workspace_bytes(int64_t n);

/* Asynchronous sem_schedule_cost: a caller-owned DEVICE workspace of at least
 * sem_cost_workspace_bytes(n) bytes (256-byte aligned) and the stream;
 * allocates nothing, does not synchronise; range errors are returned by
 * sem_check(workspace, stream). */
int sem_schedule_cost_async(const uint8_t *priority, const int32_t *prompt,
                            const int32_t *output, const int32_t *decoded, int64_t n,
                            const sem_cost_model *model, int32_t *order_out,
                            int64_t *wait_out, sem_i128 *totals_out, int32_t *service_out,
                            void *workspace, size_t ws_bytes, void *stream);

/*
 * Stage-aware selection of the next batch (Algorithm 2, blocking). Every
 * request has the key (priority, length, id) of the schedule and a stage
 * (0 = prefill, 1 = decoding):
 *   priority, length, stage [n_ids] DEVICE, indexed by request id;
 *   heap_order [n_heap] DEVICE: the waiting requests in schedule order (as
 *     sem_schedule / sem_insert return them; only the first b are read);
 *   buffer [n_buffer] DEVICE: waiting requests not yet in that schedule;
 *   ongoing [n_ongoing] DEVICE: the requests of the running batch.
 * The three lists hold distinct ids (a request is in one place only).
 * C = the b smallest keys among heap and buffer. If the smallest key of C
 * and the ongoing requests is in the prefill stage, M = C and the ongoing
 * requests merged by key; otherwise M = C's decoding members and the ongoing
 * requests, and C's prefill members are pushed back. The next batch is M's
 * first b; the rest of M is pushed back too.
 *   batch_out [b] DEVICE: the next batch in key order;
 *   pushed_out [b + n_ongoing] DEVICE: the pushed-back requests in key order;
 *   counts_out [2] int64 DEVICE: batch size, pushed-back count.
 * Sizes up to SEM_SELECT_CAP (b, n_buffer and n_ongoing each) run in one
 * workgroup's LDS; larger ones sort the lists in chunks and merge them in
 * the workspace (a few kernels more, no limit below SEM_WIDE_MAX).
 * Errors: SEM_EINVAL (negative sizes, null pointers, an id outside
 * [0, n_ids)), SEM_ENOTIMPL (min(b, n_heap) + n_buffer + n_ongoing above
 * SEM_WIDE_MAX).
 */
#define SEM_SELECT_CAP 4096
#define SEM_WIDE_MAX (1LL << 30)
int sem_select_batch(const uint8_t *priority, const int32_t *length, const uint8_t *stage,
                     int64_t n_ids, const int32_t *heap_order, int64_t n_heap,
                     const int32_t *buffer, int64_t n_buffer, const int32_t *ongoing,
                     int64_t n_ongoing, int64_t b, int32_t *batch_out, int32_t *pushed_out,
                     int64_t *counts_out);

/* Workspace size in bytes of sem_select_batch_async: 256 up to the LDS sizes,
 * then about 24 bytes per candidate and ongoing request (0 for negative
 * sizes). */
size_t sem_select_workspace_bytes(int64_t n_heap, int64_t n_buffer, int64_t n_ongoing,
                                  int64_t b);

/* Asynchronous sem_select_batch: a DEVICE workspace of at least
 * sem_select_workspace_bytes(n_heap, n_buffer, n_ongoing, b) bytes (256-byte
 * aligned) and the stream; allocates nothing, does not synchronise; errors by
 * sem_check(workspace, stream). */
int sem_select_batch_async(const uint8_t *priority, const int32_t *length,
                           const uint8_t *stage, int64_t n_ids, const int32_t *heap_order,
                           int64_t n_heap, const int32_t *buffer, int64_t n_buffer,
                           const int32_t *ongoing, int64_t n_ongoing, int64_t b,
                           int32_t *batch_out, int32_t *pushed_out, int64_t *counts_out,
                           void *workspace, size_t ws_bytes, void *stream);

/*
 * Priority-based eviction (Algorithms 3 and 4, blocking). The cached
 * requests leave the device in the inverse of the schedule order (least
 * urgent rank first, then longest remaining time, then the later arrival).
 * For incoming requests j = 0, 1, ... with KV demands demands[j], request j
 * evicts until its demand fits: victims are the shortest prefix of that
 * order whose KV sizes cover usage + (demands 0..j) - capacity (all cached
 * requests if they do not). Incoming requests are not victims of each other.
 *   priority, length [n_ids] DEVICE; cached [n_cached] int32 ids (distinct)
 *   and kv [n_cached] int64 sizes DEVICE; demands [n_demands] int64 DEVICE;
 *   victims_out [n_cached] DEVICE: the first upto_out[n_demands-1] entries
 *     receive the victims in eviction order;
 *   upto_out [n_demands] int64 DEVICE: victims after each incoming request.
 * Sums of usage and demands must stay below 2^63. Up to SEM_EVICT_CAP
 * cached requests are sorted in one workgroup's LDS; more are sorted in
 * chunks and merged in the workspace.
 * Errors: SEM_EINVAL (negative sizes, null pointers, an id outside [0, n_ids)),
 * SEM_ERANGE (a negative KV size or demand), SEM_ENOTIMPL (n_cached above
 * SEM_WIDE_MAX).
 */
#define SEM_EVICT_CAP 8192
int sem_evict(const uint8_t *priority, const int32_t *length, int64_t n_ids,
              const int32_t *cached, const int64_t *kv, int64_t n_cached, int64_t usage,
              int64_t capacity, const int64_t *demands, int64_t n_demands,
              int32_t *victims_out, int64_t *upto_out);

/* Workspace size in bytes of sem_evict_async: 256 up to SEM_EVICT_CAP cached
 * requests, then about 36 bytes per cached request (0 for n_cached < 0). */
size_t sem_evict_workspace_bytes(int64_t n_cached);

/* Asynchronous sem_evict: a DEVICE workspace of at least
 * sem_evict_workspace_bytes(n_cached) bytes (256-byte aligned) and the
 * stream; allocates nothing, does not synchronise; errors by sem_check. */
int sem_evict_async(const uint8_t *priority, const int32_t *length, int64_t n_ids,
                    const int32_t *cached, const int64_t *kv, int64_t n_cached, int64_t usage,
                    int64_t capacity, const int64_t *demands, int64_t n_demands,
                    int32_t *victims_out, int64_t *upto_out, void *workspace, size_t ws_bytes,
                    void *stream);

/*
 * Allocation-free single-queue schedule, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc. Same computation, arguments and outputs as
 * sem_schedule_async, but the workspace is a scratch array that the library
 * holds in static device memory (SEM_STATIC_SCRATCH_BYTES on every device it
 * runs on, until the process ends), so nothing is allocated or freed and the
 * call does not synchronise.
 *   status_out [1] int32 DEVICE: receives, on the stream after the schedule,
 *             SEM_OK or the device-detected error (SEM_ERANGE for a negative
 *             length).
 *   stream    the stream to enqueue on (NULL = null stream).
 * Errors returned at once: as sem_schedule_async (SEM_EINVAL also for a null
 * status_out), and SEM_ENOMEM for n > SEM_STATIC_MAX_N (the scratch holds the
 * workspace of at most that many requests).
 * All calls on one device share its scratch array: calls whose work overlaps
 * on that device (on different streams, or from different threads without
 * ordering) race and give unspecified results. Calls enqueued on one stream
 * are ordered and safe; each call clears what it needs.
 */
#define SEM_STATIC_MAX_N 1048576
#define SEM_STATIC_SCRATCH_BYTES 33554432
int sem_schedule_static(const uint8_t *priority, const int32_t *length, int64_t n,
                        int32_t *order_out, int64_t *wait_out, sem_i128 *totals_out,
                        int32_t *status_out, void *stream);

/* Stream used by the blocking calls (NULL = null stream). */
int sem_set_stream(void *stream);

/*
 * Synchronise `stream` and return the status recorded in `workspace` by the
 * last asynchronous call that used it (SEM_OK, SEM_ERANGE or SEM_EINVAL).
 */
int sem_check(const void *workspace, void *stream);

/* Static description of an error code. */
const char *sem_strerror(int code);

/*
 * Measurement hook. Arms a one-shot pair of events for one stage: the next
 * call that runs that stage records `before` and `after` (hipEvent_t passed
 * as void *, created by the caller) on its stream right before and right
 * after the stage's kernels, then disarms the stage.
 *   stage: SEM_STAGE_HIST  (multi-pass single-queue path, n > SEM_SEGMENT_CAP:
 *                           range check + first-digit histogram),
 *          SEM_STAGE_FIRST (same path: first scatter pass),
 *          SEM_STAGE_FINAL (same path: final scatter pass: order, waits, totals),
 *          SEM_STAGE_MERGE (sem_insert / sem_insert_async: the merge pass that
 *                           moves the earlier entries and places the arrivals),
 *          SEM_STAGE_POLICY (sem_schedule_policy*: for FCFS and HPJF the pass
 *                           that writes order and waits, for SJF the pass
 *                           that sums the waits per class),
 *          SEM_STAGE_COST  (sem_schedule_cost*: the service-time pass),
 *          SEM_STAGE_MID   (multi-pass path: the middle scatter passes that keys
 *                           wider than two digits need; for narrower keys one
 *                           launch that returns at once).
 * Passing NULL events disarms the stage. Returns SEM_EINVAL for an unknown
 * stage. The events are owned by the caller and must outlive the call.
 */
#define SEM_STAGE_HIST 0
#define SEM_STAGE_FIRST 1
#define SEM_STAGE_FINAL 2
#define SEM_STAGE_MERGE 3
#define SEM_STAGE_POLICY 4
#define SEM_STAGE_COST 5
#define SEM_STAGE_MID 6
int sem_trace_stage(int stage, void *before, void *after);

#ifdef __cplusplus
}
#endif

#endif /* SEMSCHED_H */
