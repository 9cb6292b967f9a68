/*
 * CPU oracle for the semantic-scheduling hot path (plain C).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link or call
 * this file: only the tests, the smoke check and the benchmark's CPU
 * baseline load it. It shares no code, header or table with the HIP library.
 *
 * The computation is the plain definition, the same as the pure-Python
 * oracle (semsched_oracle.py), written for speed on large queues:
 *
 *   1. order: ids ascending by (rank p, predicted length l, id), i.e. the
 *      drained min-heap keyed by the priority tuple (f_e, f_t) of
 *      Algorithm 1 (MinHeap Construction); the id breaks exact ties
 *      (the paper gives no tie rule).
 *   2. wait[0] = 0, wait[k] = wait[k-1] + l[order[k-1]]  (exclusive prefix of
 *      service times ahead of each request; Eq. 1 with equal arrivals).
 *   3. totals[0] = sum of waits; totals[1+c] = sum over requests of class c.
 *      Exact 128-bit (unsigned __int128), split into lo/hi words.
 *
 * The sort is a top-down merge sort on (p, l, id) records. Because the
 * comparison covers the id, the order is total and any correct sort gives
 * the same permutation.
 *
 * oracle_schedule_policy orders by the comparison policies of Section 4
 * instead (arrival order; length then id; rank then id); waits and
 * per-class totals are defined the same way for every policy.
 */
#include <stdint.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ERANGE (-2)
#define ORACLE_ENOMEM (-3)

typedef struct {
  int32_t len;
  int32_t id;
  uint8_t pri;
} rec_t;

/* Comparison policies of the experiments (Section 4): which fields key the
 * order before the id. 0 = (rank, length), 1 = none (arrival order),
 * 2 = (length), 3 = (rank). */
#define ORACLE_POLICY_SEMANTIC 0
#define ORACLE_POLICY_FCFS 1
#define ORACLE_POLICY_SJF 2
#define ORACLE_POLICY_HPJF 3

static int rec_less(const rec_t *a, const rec_t *b, int policy) {
  const int use_pri = policy == ORACLE_POLICY_SEMANTIC || policy == ORACLE_POLICY_HPJF;
  const int use_len = policy == ORACLE_POLICY_SEMANTIC || policy == ORACLE_POLICY_SJF;
  if (use_pri && a->pri != b->pri) return a->pri < b->pri;
  if (use_len && a->len != b->len) return a->len < b->len;
  return a->id < b->id;
}

static void merge_sort(rec_t *a, rec_t *tmp, int64_t n, int policy) {
  if (n < 2) return;
  int64_t h = n / 2;
  merge_sort(a, tmp, h, policy);
  merge_sort(a + h, tmp, n - h, policy);
  int64_t i = 0, j = h, k = 0;
  while (i < h && j < n) {
    if (rec_less(&a[j], &a[i], policy))
      tmp[k++] = a[j++];
    else
      tmp[k++] = a[i++];
  }
  while (i < h) tmp[k++] = a[i++];
  while (j < n) tmp[k++] = a[j++];
  memcpy(a, tmp, (size_t)n * sizeof(rec_t));
}

/* One queue. totals_lo/hi have 1 + num_classes entries. */
static int schedule_one(const uint8_t *pri, const int32_t *len, int64_t n,
                        int32_t num_classes, int policy, int32_t *order,
                        int64_t *wait, uint64_t *totals_lo, uint64_t *totals_hi,
                        rec_t *recs, rec_t *tmp) {
  for (int64_t i = 0; i < n; ++i) {
    if (len[i] < 0 || (int32_t)pri[i] >= num_classes) return ORACLE_ERANGE;
    recs[i].pri = pri[i];
    recs[i].len = len[i];
    recs[i].id = (int32_t)i;
  }
  merge_sort(recs, tmp, n, policy);

  unsigned __int128 tot[257];
  for (int c = 0; c <= num_classes; ++c) tot[c] = 0;
  int64_t running = 0;
  for (int64_t k = 0; k < n; ++k) {
    order[k] = recs[k].id;
    wait[k] = running;
    tot[0] += (unsigned __int128)(uint64_t)running;
    tot[1 + recs[k].pri] += (unsigned __int128)(uint64_t)running;
    running += recs[k].len;
  }
  for (int c = 0; c <= num_classes; ++c) {
    totals_lo[c] = (uint64_t)tot[c];
    totals_hi[c] = (uint64_t)(tot[c] >> 64);
  }
  return ORACLE_OK;
}

int oracle_schedule_policy(int policy, const uint8_t *pri, const int32_t *len,
                           int64_t n, int32_t *order, int64_t *wait,
                           uint64_t *totals_lo, uint64_t *totals_hi) {
  if (n < 0 || n > INT32_MAX) return ORACLE_EINVAL;
  if (policy < ORACLE_POLICY_SEMANTIC || policy > ORACLE_POLICY_HPJF) return ORACLE_EINVAL;
  rec_t *recs = (rec_t *)malloc((size_t)(n ? n : 1) * sizeof(rec_t));
  rec_t *tmp = (rec_t *)malloc((size_t)(n ? n : 1) * sizeof(rec_t));
  if (!recs || !tmp) {
    free(recs);
    free(tmp);
    return ORACLE_ENOMEM;
  }
  int rc = schedule_one(pri, len, n, 256, policy, order, wait, totals_lo,
                        totals_hi, recs, tmp);
  free(recs);
  free(tmp);
  return rc;
}

int oracle_schedule(const uint8_t *pri, const int32_t *len, int64_t n,
                    int32_t *order, int64_t *wait, uint64_t *totals_lo,
                    uint64_t *totals_hi) {
  return oracle_schedule_policy(ORACLE_POLICY_SEMANTIC, pri, len, n, order,
                                wait, totals_lo, totals_hi);
}

int oracle_schedule_batched(const uint8_t *pri, const int32_t *len,
                            const int64_t *offsets, int64_t num_segments,
                            int32_t num_classes, int32_t *order, int64_t *wait,
                            uint64_t *totals_lo, uint64_t *totals_hi) {
  if (num_segments < 0 || num_classes < 1 || num_classes > 256)
    return ORACLE_EINVAL;
  if (offsets[0] != 0) return ORACLE_EINVAL;
  int64_t biggest = 0;
  for (int64_t s = 0; s < num_segments; ++s) {
    int64_t m = offsets[s + 1] - offsets[s];
    if (m < 0 || m > INT32_MAX) return ORACLE_EINVAL;
    if (m > biggest) biggest = m;
  }
  rec_t *recs = (rec_t *)malloc((size_t)(biggest ? biggest : 1) * sizeof(rec_t));
  rec_t *tmp = (rec_t *)malloc((size_t)(biggest ? biggest : 1) * sizeof(rec_t));
  if (!recs || !tmp) {
    free(recs);
    free(tmp);
    return ORACLE_ENOMEM;
  }
  int rc = ORACLE_OK;
  const int64_t stride = 1 + num_classes;
  for (int64_t s = 0; s < num_segments && rc == ORACLE_OK; ++s) {
    int64_t a = offsets[s], m = offsets[s + 1] - offsets[s];
    rc = schedule_one(pri + a, len + a, m, num_classes, ORACLE_POLICY_SEMANTIC,
                      order + a, wait + a,
                      totals_lo + s * stride, totals_hi + s * stride, recs, tmp);
  }
  free(recs);
  free(tmp);
  return rc;
}

/*
 * The same schedule of independent queues with the queues spread over the
 * host's threads (OpenMP): each thread runs the per-queue routine above on
 * whole queues, with buffers of its own. Only the CPU baseline of the
 * batched workloads uses it; the arithmetic is schedule_one's.
 */
int oracle_schedule_batched_parallel(const uint8_t *pri, const int32_t *len,
                                     const int64_t *offsets, int64_t num_segments,
                                     int32_t num_classes, int32_t *order, int64_t *wait,
                                     uint64_t *totals_lo, uint64_t *totals_hi,
                                     int32_t *threads_used) {
  if (num_segments < 0 || num_classes < 1 || num_classes > 256)
    return ORACLE_EINVAL;
  if (offsets[0] != 0) return ORACLE_EINVAL;
  int64_t biggest = 0;
  for (int64_t s = 0; s < num_segments; ++s) {
    int64_t m = offsets[s + 1] - offsets[s];
    if (m < 0 || m > INT32_MAX) return ORACLE_EINVAL;
    if (m > biggest) biggest = m;
  }
  const int64_t stride = 1 + num_classes;
  int rc = ORACLE_OK;
  int used = 1;
  /* queues handed out in chunks of up to 16, fewer when there are too few
     queues to give every thread several chunks (16 long queues: one each) */
  const int64_t per = num_segments / (8 * (int64_t)omp_get_max_threads());
  const int chunk = (int)(per < 1 ? 1 : (per > 16 ? 16 : per));
#pragma omp parallel
  {
    rec_t *recs = (rec_t *)malloc((size_t)(biggest ? biggest : 1) * sizeof(rec_t));
    rec_t *tmp = (rec_t *)malloc((size_t)(biggest ? biggest : 1) * sizeof(rec_t));
    int mine = (recs && tmp) ? ORACLE_OK : ORACLE_ENOMEM;
#pragma omp single
    used = omp_get_num_threads();
#pragma omp for schedule(dynamic, chunk)
    for (int64_t s = 0; s < num_segments; ++s) {
      if (mine != ORACLE_OK) continue;
      int64_t a = offsets[s], m = offsets[s + 1] - offsets[s];
      int r = schedule_one(pri + a, len + a, m, num_classes, ORACLE_POLICY_SEMANTIC,
                           order + a, wait + a, totals_lo + s * stride,
                           totals_hi + s * stride, recs, tmp);
      if (r != ORACLE_OK) mine = r;
    }
#pragma omp critical
    if (mine != ORACLE_OK) rc = mine;
    free(recs);
    free(tmp);
  }
  if (threads_used) *threads_used = used;
  return rc;
}

/*
 * Cost model of Section 3.4 (the same definitions and readings as
 * cost_oracle.py): constants are Q32.32 integers {alpha1, alpha2, beta,
 * gamma1, gamma2}; every product and sum is exact in unsigned __int128.
 */
typedef unsigned __int128 u128;

/* a + b, setting *over when the sum passes 2^128 (the service time then
 * saturates). */
static u128 add_q(u128 a, u128 b, int *over) {
  const u128 s = a + b;
  if (s < a) *over = 1;
  return s;
}

static u128 decode_cost_q(const uint64_t *c, u128 n, u128 m, int *over) {
  return add_q((u128)c[3] * ((m * m + m) / 2 + n * m), (u128)c[4] * m, over);
}

int oracle_service_times(const int32_t *prompt, const int32_t *output,
                         const int32_t *decoded, int64_t n, const uint64_t *c,
                         int32_t *out) {
  if (n < 0) return ORACLE_EINVAL;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t a = prompt[i], m = output[i], d = decoded ? decoded[i] : 0;
    if (a < 0 || m < 0 || d < 0) return ORACLE_ERANGE;
    const int64_t r = m > d ? m - d : 0;
    int over = 0;
    u128 cost = decode_cost_q(c, (u128)(a + d), (u128)r, &over);
    if (d == 0) {
      cost = add_q(cost, (u128)c[0] * (u128)a * (u128)a, &over);
      cost = add_q(cost, (u128)c[1] * (u128)a, &over);
    }
    const u128 s = cost >> 32;
    out[i] = (over || s > (u128)INT32_MAX) ? INT32_MAX : (int32_t)s;
  }
  return ORACLE_OK;
}

int oracle_evict_plan(const int32_t *prompt, const int32_t *decoded, int64_t n,
                      const uint64_t *c, uint8_t *keep, int32_t *save) {
  if (n < 0) return ORACLE_EINVAL;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t a = prompt[i], mp = decoded[i];
    if (a < 0 || mp < 0) return ORACLE_ERANGE;
    const u128 reload = (u128)c[2] * (u128)a;
    int over = 0;
    const u128 recompute = add_q((u128)c[0] * (u128)a * (u128)a, (u128)c[1] * (u128)a, &over);
    keep[i] = (over || reload < recompute) ? 1 : 0;
    /* first y whose next recomputed token does not pay: gamma1*(y+1+n)+gamma2 >= beta */
    int64_t y = 0;
    while (y < mp && (u128)c[3] * (u128)(y + 1 + a) + (u128)c[4] < (u128)c[2]) ++y;
    save[i] = (int32_t)(mp - y);
  }
  return ORACLE_OK;
}
