/*
 * hbf_oracle.c -- plain, slow, sequential CPU reference of the HBF service
 * model.  TEST INFRASTRUCTURE ONLY: nothing in the product path may link,
 * load or call this file; only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg do.  It shares no code, header, constant or
 * table with the HIP implementation.
 *
 * What it computes (paper: HBFSim, arXiv 2609.09800):
 *  - Explicit range registration and fail-closed classification of an
 *    address against the sorted snapshot of registered ranges
 *    (Section "D1: An Explicit and Fail-Closed Boundary").  An address
 *    outside every range takes the native path: zero modeled delay.
 *  - Each in-range access becomes one foreground media request (a page
 *    read) that is timed by an online media model (Section "Design",
 *    opening paragraph: each foreground request is placed into the online
 *    media-model instance and its completion is returned to the request).
 *    The paper delegates the media model to MQSim and publishes no timing
 *    parameters (Section "Motivation": the specification defers every
 *    time quantity to vendor datasheets).  This oracle therefore takes the
 *    reading used throughout the project: a die-read stage (service tR,
 *    FCFS in (issue, index) order, one queue per die) followed by a
 *    channel-transfer stage (service xfer, FCFS in (die-done, index) order,
 *    one queue per channel), both with infinite buffers and resource clocks
 *    that persist across calls.
 *
 * Readings where the paper is silent (each is a documented choice):
 *  - address -> device page: p = dev_page_base(range) + (addr-base)/page,
 *    dev_page_base = pages of earlier-registered ranges, in registration
 *    order.
 *  - page -> (channel, die, plane, page-in-plane): channel-first striping,
 *    ch = p mod C, die = (p / C) mod D, plane = (p / (C*D)) mod P,
 *    pg = p / (C*D*P).
 *  - die queue key = (ch, die); with the plane-parallel flag (ch, die, plane).
 *  - media variant (flag): die page-register blocking, see
 *    orc_blocking_stage.
 *  - timing source (flag): the calibrated end-to-end vmem burst curve
 *    instead of the media model, see orc_vmem_stage.
 *  - xfer = ceil(page_bytes * 1e9 / channel_bytes_per_s) in integer ns.
 *  - times are int64 ns; "idle since minus infinity" at create/reset.
 *
 * Every step below is written in the order the model defines it, with no
 * blocking, fusion or reordering: validate, classify, map, die stage in
 * request order, sort by (die_done, index), channel stage in that order.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* Status codes of the public contract (values fixed by the C ABI docs). */
#define ORC_OK             0
#define ORC_EINVAL        -1
#define ORC_EALIGN        -2
#define ORC_EOVERLAP      -3
#define ORC_ENOWORKSPACE  -4
#define ORC_EUNSORTED     -5
#define ORC_ERANGE_TIME   -6
#define ORC_EHIP          -7
#define ORC_ENOMEM        -8

#define ORC_TIME_ERROR    INT64_MIN
#define ORC_FLAG_PLANE_PARALLEL 1u
#define ORC_FLAG_REGISTER_BLOCKING 2u
#define ORC_FLAG_VMEM_CURVE 4u
#define ORC_MAX_RANGES    64

/* Issue times must lie in [0, 2^61); any modeled time reaching 2^62 is an
 * overflow of the model's time domain and fails the whole call. */
#define ORC_ISSUE_LIMIT   ((int64_t)1 << 61)
#define ORC_TIME_LIMIT    ((int64_t)1 << 62)
#define ORC_SERVICE_LIMIT ((int64_t)1 << 29)
#define ORC_N_LIMIT       ((int64_t)1 << 31)

typedef struct {
  uint32_t channels, dies_per_channel, planes_per_die, page_bytes;
  int64_t  t_read_ns;
  uint64_t channel_bytes_per_s;
  uint32_t flags;
} orc_params;

typedef struct {
  uint64_t base, bytes, dev_page_base;
} orc_range;

typedef struct {
  orc_params p;
  int64_t xfer_ns;
  int n_ranges;
  orc_range ranges[ORC_MAX_RANGES];   /* in registration order */
  uint64_t total_pages;
  int64_t *die_free;    /* per die queue key; idle = has_die_free 0 */
  uint8_t *die_busy;    /* 0 = idle since -inf */
  int64_t *chan_free;
  uint8_t *chan_busy;
  uint32_t n_die_keys;
  /* refresh (Section D4): per die queue, the ids of its pending quanta in
   * plan order; the completion time of every quantum ever submitted */
  int64_t t_prog_ns;
  struct orc_fifo *fifo;
  int64_t *qdone;
  int64_t nq, qcap;
  /* vmem curve: burst cost at the knots, the route's clock, the device
   * page of the last access and the length of the burst it ended */
  int64_t vknot[6];
  int64_t vfree;
  uint8_t vbusy, vhave;
  uint64_t vlast;
  int64_t vburst;
} orc_model;

typedef struct orc_fifo { int64_t *id; int64_t head, len, cap; } orc_fifo;
#define ORC_REFRESH_PENDING ((int64_t)-1)

uint32_t orc_n_die_keys(const orc_params *p) {
  uint64_t k = (uint64_t)p->channels * p->dies_per_channel;
  if (p->flags & ORC_FLAG_PLANE_PARALLEL) k *= p->planes_per_die;
  return (uint32_t)k;
}

int orc_create(const orc_params *p, orc_model **out) {
  if (!p || !out) return ORC_EINVAL;
  if (p->channels == 0 || p->dies_per_channel == 0 || p->planes_per_die == 0) return ORC_EINVAL;
  if (p->page_bytes == 0) return ORC_EINVAL;
  if (p->t_read_ns < 1 || p->t_read_ns > ORC_SERVICE_LIMIT) return ORC_EINVAL;
  if (p->channel_bytes_per_s == 0) return ORC_EINVAL;
  if (p->flags & ~(ORC_FLAG_PLANE_PARALLEL | ORC_FLAG_REGISTER_BLOCKING | ORC_FLAG_VMEM_CURVE)) return ORC_EINVAL;
  if ((p->flags & ORC_FLAG_VMEM_CURVE) && (p->flags & ORC_FLAG_REGISTER_BLOCKING)) return ORC_EINVAL;
  if ((uint64_t)p->channels * p->dies_per_channel * p->planes_per_die > 65536u) return ORC_EINVAL;
  /* transfer time: ceil(page_bytes * 1e9 / bytes_per_s), exact integers */
  unsigned __int128 num = (unsigned __int128)p->page_bytes * 1000000000u;
  unsigned __int128 q = (num + p->channel_bytes_per_s - 1) / p->channel_bytes_per_s;
  if (q < 1 || q > (unsigned __int128)ORC_SERVICE_LIMIT) return ORC_EINVAL;
  orc_model *m = (orc_model *)calloc(1, sizeof(orc_model));
  if (!m) return ORC_ENOMEM;
  m->p = *p;
  m->xfer_ns = (int64_t)q;
  /* vmem curve until configured: every page of a burst costs the
   * single-page value the paper prints (11,133 ns), i.e. no burst benefit */
  for (int k = 0; k < 6; k++) m->vknot[k] = 11133 * (int64_t[]){1, 4, 16, 64, 256, 512}[k];
  m->n_die_keys = orc_n_die_keys(p);
  m->die_free = (int64_t *)calloc(m->n_die_keys, sizeof(int64_t));
  m->die_busy = (uint8_t *)calloc(m->n_die_keys, 1);
  m->chan_free = (int64_t *)calloc(p->channels, sizeof(int64_t));
  m->chan_busy = (uint8_t *)calloc(p->channels, 1);
  if (!m->die_free || !m->die_busy || !m->chan_free || !m->chan_busy) {
    free(m->die_free); free(m->die_busy); free(m->chan_free); free(m->chan_busy); free(m);
    return ORC_ENOMEM;
  }
  *out = m;
  return ORC_OK;
}

void orc_destroy(orc_model *m) {
  if (!m) return;
  if (m->fifo)
    for (uint32_t k = 0; k < m->n_die_keys; k++) free(m->fifo[k].id);
  free(m->fifo); free(m->qdone);
  free(m->die_free); free(m->die_busy); free(m->chan_free); free(m->chan_busy);
  free(m);
}

int64_t orc_xfer_ns(const orc_model *m) { return m->xfer_ns; }

/* Return every resource to "idle since minus infinity". */
void orc_reset(orc_model *m) {
  /* pending refresh quanta are dropped; their completion stays pending */
  if (m->fifo)
    for (uint32_t k = 0; k < m->n_die_keys; k++) m->fifo[k].head = m->fifo[k].len = 0;
  memset(m->die_busy, 0, m->n_die_keys);
  memset(m->chan_busy, 0, m->p.channels);
  memset(m->die_free, 0, sizeof(int64_t) * m->n_die_keys);
  memset(m->chan_free, 0, sizeof(int64_t) * m->p.channels);
  m->vfree = 0;
  m->vbusy = 0;
  m->vhave = 0;
  m->vlast = 0;
  m->vburst = 0;
}

/* Range registration (Section D1): explicit [base, base+bytes) intervals,
 * page aligned, never overlapping. */
int orc_register_range(orc_model *m, uint64_t base, uint64_t bytes) {
  if (!m || bytes == 0) return ORC_EINVAL;
  if (m->n_ranges >= ORC_MAX_RANGES) return ORC_EINVAL;
  if (base % m->p.page_bytes != 0 || bytes % m->p.page_bytes != 0) return ORC_EALIGN;
  if (base + bytes < base) return ORC_EINVAL;             /* wraps past 2^64 */
  for (int r = 0; r < m->n_ranges; r++) {
    uint64_t b = m->ranges[r].base, e = m->ranges[r].base + m->ranges[r].bytes;
    if (base < e && b < base + bytes) return ORC_EOVERLAP;
  }
  m->ranges[m->n_ranges].base = base;
  m->ranges[m->n_ranges].bytes = bytes;
  m->ranges[m->n_ranges].dev_page_base = m->total_pages;
  m->total_pages += bytes / m->p.page_bytes;
  m->n_ranges++;
  return ORC_OK;
}

/* Classification (Section D1): the index of the range containing addr, or
 * -1 for the native path.  A linear scan is the plain definition. */
static int orc_classify(const orc_model *m, uint64_t addr) {
  for (int r = 0; r < m->n_ranges; r++)
    if (addr >= m->ranges[r].base && addr - m->ranges[r].base < m->ranges[r].bytes) return r;
  return -1;
}

typedef struct { uint32_t ch, die, plane; uint64_t page; uint32_t key; } orc_loc;

/* (channel, die, plane, page) of device page dp by channel-first striping. */
static orc_loc orc_locate(const orc_model *m, uint64_t dp) {
  const orc_params *p = &m->p;
  orc_loc L;
  L.ch = (uint32_t)(dp % p->channels);
  L.die = (uint32_t)((dp / p->channels) % p->dies_per_channel);
  L.plane = (uint32_t)((dp / ((uint64_t)p->channels * p->dies_per_channel)) % p->planes_per_die);
  L.page = dp / ((uint64_t)p->channels * p->dies_per_channel * p->planes_per_die);
  L.key = L.ch * p->dies_per_channel + L.die;
  if (p->flags & ORC_FLAG_PLANE_PARALLEL) L.key = L.key * p->planes_per_die + L.plane;
  return L;
}

/* Device page of addr in range r, and its location. */
static orc_loc orc_map(const orc_model *m, int r, uint64_t addr) {
  return orc_locate(m, m->ranges[r].dev_page_base + (addr - m->ranges[r].base) / m->p.page_bytes);
}

/* Packed classification word (documented format of hbf_classify_map):
 * bit 63 in-range; bits 62..56 range index; 55..50 plane; 49..42 die;
 * 41..32 channel; 31..0 page within the plane.  Out of range: 0. */
static uint64_t orc_pack(int r, orc_loc L) {
  return (1ull << 63) | ((uint64_t)r << 56) | ((uint64_t)L.plane << 50) |
         ((uint64_t)L.die << 42) | ((uint64_t)L.ch << 32) | (L.page & 0xffffffffull);
}

int orc_classify_map(const orc_model *m, const uint64_t *addr, int64_t n, uint64_t *map_out) {
  if (!m || n < 0 || (n > 0 && (!addr || !map_out))) return ORC_EINVAL;
  const orc_params *p = &m->p;
  if (p->channels > 1024 || p->dies_per_channel > 256 || p->planes_per_die > 64) return ORC_EINVAL;
  for (int64_t i = 0; i < n; i++) {
    int r = orc_classify(m, addr[i]);
    if (r < 0) { map_out[i] = 0; continue; }
    orc_loc L = orc_map(m, r, addr[i]);
    if (L.page > 0xffffffffull) return ORC_EINVAL;
    map_out[i] = orc_pack(r, L);
  }
  return ORC_OK;
}

typedef struct { int64_t dd; int64_t idx; } orc_pair;

static int orc_cmp_pair(const void *a, const void *b) {
  const orc_pair *x = (const orc_pair *)a, *y = (const orc_pair *)b;
  if (x->dd != y->dd) return x->dd < y->dd ? -1 : 1;
  if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
  return 0;
}

static int64_t orc_max(int64_t a, int64_t b) { return a > b ? a : b; }

/*
 * Media variant: die page-register blocking.  A die queue holds one page
 * register: a read leaves its page there, and the die's next read may start
 * only once that page has left the register, i.e. once its channel transfer
 * has completed.  The channel still serves pages FCFS by (die-done, index).
 * Each channel and its die queues are simulated in service order: at every
 * step the pending page with the smallest (die-done, index) among the
 * channel's die queues is transferred, which frees its die for the next
 * read (each die queue has at most one page pending).  Refresh claims follow
 * the same rule as without blocking (a claim adds tQ before the read).
 * Returns 1 on a time-domain overflow.
 */
static int orc_blocking_stage(orc_model *m, const int64_t *issue, int64_t n, int8_t *in, const uint32_t *key,
                              const uint32_t *chan, int64_t *dd, int64_t *complete, int64_t *df, uint8_t *db,
                              int64_t *cf, uint8_t *cb, int64_t *claimed, int64_t tQ, int *nomem) {
  const uint32_t K = m->n_die_keys, C = m->p.channels, Dk = K / C;
  const int64_t tR = m->p.t_read_ns, xfer = m->xfer_ns;
  int64_t *start = (int64_t *)calloc((size_t)K + 1, sizeof(int64_t));
  int64_t *head = (int64_t *)calloc((size_t)K, sizeof(int64_t));
  int64_t *list = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n ? n : 1));
  if (!start || !head || !list) { free(start); free(head); free(list); *nomem = 1; return 0; }
  (void)chan;
  /* each die queue's requests in index order (= FCFS) */
  for (int64_t i = 0; i < n; i++)
    if (in[i]) start[key[i] + 1]++;
  for (uint32_t k = 0; k < K; k++) start[k + 1] += start[k];
  for (uint32_t k = 0; k < K; k++) head[k] = start[k];
  for (int64_t i = 0; i < n; i++)
    if (in[i]) list[head[key[i]]++] = i;
  for (uint32_t k = 0; k < K; k++) head[k] = start[k];
  int overflow = 0;
  for (uint32_t c = 0; c < C; c++) {
    /* admit the first request of every die queue of the channel */
    for (uint32_t k = c * Dk; k < (c + 1) * Dk; k++) {
      if (head[k] == start[k + 1]) continue;
      const int64_t i = list[head[k]];
      int64_t s0 = db[k] ? orc_max(issue[i], df[k]) : issue[i];
      if (m->fifo && claimed[k] < m->fifo[k].len - m->fifo[k].head) { claimed[k]++; in[i] = 2; s0 += tQ; }
      dd[i] = s0 + tR;
      if (dd[i] >= ORC_TIME_LIMIT) overflow = 1;
    }
    for (;;) {
      /* the pending page that reached the channel first: smallest (dd, index) */
      int64_t best = -1;
      uint32_t bk = 0;
      for (uint32_t k = c * Dk; k < (c + 1) * Dk; k++) {
        if (head[k] == start[k + 1]) continue;
        const int64_t i = list[head[k]];
        if (best < 0 || dd[i] < dd[best] || (dd[i] == dd[best] && i < best)) { best = i; bk = k; }
      }
      if (best < 0) break;
      const int64_t s1 = cb[c] ? orc_max(dd[best], cf[c]) : dd[best];
      complete[best] = s1 + xfer;
      if (complete[best] >= ORC_TIME_LIMIT) overflow = 1;
      cf[c] = complete[best];
      cb[c] = 1;
      /* the page has left the register: the die may read again */
      df[bk] = complete[best];
      db[bk] = 1;
      head[bk]++;
      if (head[bk] < start[bk + 1]) {
        const int64_t i = list[head[bk]];
        int64_t s0 = orc_max(issue[i], complete[best]);
        if (m->fifo && claimed[bk] < m->fifo[bk].len - m->fifo[bk].head) { claimed[bk]++; in[i] = 2; s0 += tQ; }
        dd[i] = s0 + tR;
        if (dd[i] >= ORC_TIME_LIMIT) overflow = 1;
      }
      if (overflow) break;   /* the call fails; the rest does not matter */
    }
    if (overflow) break;
  }
  free(start); free(head); free(list);
  return overflow;
}

/* ---------------------------------------------------------------- vmem curve
 * Section "Discussion": a second timing source, a calibrated end-to-end curve
 * measured on a host paging path that presents an SSD as memory.  The curve
 * prices a sequential burst of L pages; its knots are at 1, 4, 16, 64, 256
 * and 512 pages, and beyond the last knot it keeps the final segment's slope.
 * An access that jumps elsewhere, steps back, re-reads the same page or
 * switches operation does not extend a burst: it begins a fresh one-page
 * burst at the single-page price the paper prints, 11,133 ns.  Readings (the paper prints only that one knot value and
 * does not say how a burst becomes per-access completion times):
 *  - T(L), the cost of a burst of L pages: T(0) = 0; the six knot values are
 *    parameters (orc_vmem_configure); between knots T is linear in L,
 *    rounded down to whole ns; past 512, T(512) + floor((T(512) - T(256)) *
 *    (L - 512) / 256);
 *  - an access continues the burst iff its device page is the page right
 *    after the previous in-range access's page (request order, across calls
 *    until reset); every other access (any other page: random, reverse,
 *    repeated) starts a new burst.  Every request is a page read, so the
 *    operation never changes and no cross-operation reset arises;
 *  - the route serves one access at a time in request order: the access at
 *    burst position L occupies it for T(L) - T(L-1), so a back-to-back burst
 *    of L pages takes T(L) and a lone access T(1);
 *  - complete = max(issue, route free) + that service; the route's clock
 *    persists across calls like the media model's (idle after reset);
 *    out-of-range requests take the native path (complete = issue). */
static const int64_t ORC_VKNOT_PAGES[6] = {1, 4, 16, 64, 256, 512};

/* T(L): cost of a sequential burst of L pages. */
int64_t orc_vmem_burst_ns(const orc_model *m, int64_t L) {
  const int64_t *T = m->vknot;
  if (L <= 0) return 0;
  if (L > 512)
    return T[5] + (int64_t)((__int128)(T[5] - T[4]) * (L - 512) / 256);
  int s = 0;  /* the segment [knot s, knot s+1] holding L */
  while (s < 4 && L > ORC_VKNOT_PAGES[s + 1]) s++;
  const int64_t La = ORC_VKNOT_PAGES[s], Lb = ORC_VKNOT_PAGES[s + 1];
  return T[s] + (int64_t)((__int128)(T[s + 1] - T[s]) * (L - La) / (Lb - La));
}

/* Knot values T(1), T(4), T(16), T(64), T(256), T(512) in ns: T(1) >= 1,
 * nondecreasing, and no page of any segment (nor a lone page) costing more
 * than 2^29 ns on average. */
int orc_vmem_configure(orc_model *m, const int64_t *knot) {
  if (!m || !knot) return ORC_EINVAL;
  if (knot[0] < 1 || knot[0] > ORC_SERVICE_LIMIT) return ORC_EINVAL;
  for (int k = 1; k < 6; k++) {
    if (knot[k] < knot[k - 1]) return ORC_EINVAL;
    if (knot[k] - knot[k - 1] > ORC_SERVICE_LIMIT * (ORC_VKNOT_PAGES[k] - ORC_VKNOT_PAGES[k - 1])) return ORC_EINVAL;
  }
  for (int k = 0; k < 6; k++) m->vknot[k] = knot[k];
  return ORC_OK;
}

/* The route's state: {clock (INT64_MIN if idle), last device page (-1 if
 * none), length of the burst that page ended (0 if none)}. */
void orc_vmem_state(const orc_model *m, int64_t *out) {
  out[0] = m->vbusy ? m->vfree : INT64_MIN;
  out[1] = m->vhave ? (int64_t)m->vlast : -1;
  out[2] = m->vhave ? m->vburst : 0;
}

/* Requests in index order on the vmem route (validation done by the caller).
 * Returns 1 on a time-domain overflow (state then untouched). */
static int orc_vmem_stage(orc_model *m, const uint64_t *addr, const int64_t *issue, int64_t n,
                          int64_t *complete) {
  int64_t vf = m->vfree, L = m->vburst;
  uint8_t vb = m->vbusy, have = m->vhave;
  uint64_t last = m->vlast;
  int overflow = 0;
  for (int64_t i = 0; i < n; i++) {
    int r = orc_classify(m, addr[i]);
    if (r < 0) { complete[i] = issue[i]; continue; }
    uint64_t page = m->ranges[r].dev_page_base + (addr[i] - m->ranges[r].base) / m->p.page_bytes;
    L = (have && page == last + 1) ? L + 1 : 1;
    last = page;
    have = 1;
    int64_t service = orc_vmem_burst_ns(m, L) - orc_vmem_burst_ns(m, L - 1);
    int64_t start = vb ? orc_max(issue[i], vf) : issue[i];
    complete[i] = start + service;
    if (complete[i] >= ORC_TIME_LIMIT) overflow = 1;
    vf = complete[i];
    vb = 1;
  }
  if (overflow) return 1;
  m->vfree = vf; m->vbusy = vb; m->vhave = have; m->vlast = last; m->vburst = L;
  return 0;
}

/*
 * The timing call.  Steps, in the model's order:
 *  1. validate every issue time (0 <= t < 2^61, nondecreasing in index);
 *  2. classify + map every request;
 *  3. die stage, requests in index order (= FCFS by (issue, index)):
 *       start = max(issue, die_free), die_done = start + tR;
 *  4. sort the in-range requests by (die_done, index);
 *  5. channel stage in that order:
 *       start = max(die_done, chan_free), complete = start + xfer;
 *  6. out-of-range requests: complete = issue (native path, no delay).
 * On a validation or time-domain error every output is ORC_TIME_ERROR and the
 * resource clocks keep their values from before the call.
 */
int orc_time_requests(orc_model *m, const uint64_t *addr, const int64_t *issue, int64_t n,
                      int64_t *complete) {
  if (!m || n < 0 || n > ORC_N_LIMIT || (n > 0 && (!addr || !issue || !complete))) return ORC_EINVAL;
  if (n == 0) return ORC_OK;
  const orc_params *p = &m->p;
  const int64_t tR = p->t_read_ns, xfer = m->xfer_ns;

  /* 1. validation; a bad time range takes precedence over disorder */
  int bad_range = 0, bad_order = 0;
  for (int64_t i = 0; i < n; i++) {
    if (issue[i] < 0 || issue[i] >= ORC_ISSUE_LIMIT) bad_range = 1;
    if (i > 0 && issue[i] < issue[i - 1]) bad_order = 1;
  }
  if (bad_range || bad_order) {
    for (int64_t i = 0; i < n; i++) complete[i] = ORC_TIME_ERROR;
    return bad_range ? ORC_ERANGE_TIME : ORC_EUNSORTED;
  }
  if (p->flags & ORC_FLAG_VMEM_CURVE) {
    if (orc_vmem_stage(m, addr, issue, n, complete)) {
      for (int64_t i = 0; i < n; i++) complete[i] = ORC_TIME_ERROR;
      return ORC_ERANGE_TIME;
    }
    return ORC_OK;
  }

  /* working copies of the clocks: committed only if the call succeeds */
  int64_t *df = (int64_t *)malloc(sizeof(int64_t) * m->n_die_keys);
  uint8_t *db = (uint8_t *)malloc(m->n_die_keys);
  int64_t *cf = (int64_t *)malloc(sizeof(int64_t) * p->channels);
  uint8_t *cb = (uint8_t *)malloc(p->channels);
  int64_t *dd = (int64_t *)malloc(sizeof(int64_t) * n);
  uint32_t *chan = (uint32_t *)malloc(sizeof(uint32_t) * n);
  int8_t *in = (int8_t *)malloc(n);
  orc_pair *ord = (orc_pair *)malloc(sizeof(orc_pair) * n);
  const int blocking = (p->flags & ORC_FLAG_REGISTER_BLOCKING) != 0;
  uint32_t *key = blocking ? (uint32_t *)malloc(sizeof(uint32_t) * n) : NULL;
  if (!df || !db || !cf || !cb || !dd || !chan || !in || !ord || (blocking && !key)) {
    free(df); free(db); free(cf); free(cb); free(dd); free(chan); free(in); free(ord); free(key);
    return ORC_ENOMEM;
  }
  memcpy(df, m->die_free, sizeof(int64_t) * m->n_die_keys);
  memcpy(db, m->die_busy, m->n_die_keys);
  memcpy(cf, m->chan_free, sizeof(int64_t) * p->channels);
  memcpy(cb, m->chan_busy, p->channels);

  /* refresh claims of this call per die queue (committed with the clocks) */
  int64_t *claimed = (int64_t *)calloc(m->n_die_keys, sizeof(int64_t));
  if (!claimed) {
    free(df); free(db); free(cf); free(cb); free(dd); free(chan); free(in); free(ord); free(key);
    return ORC_ENOMEM;
  }
  const int64_t tQ = tR + m->t_prog_ns;

  int overflow = 0;
  int64_t n_in = 0;
  /* 2.+3. classify, map and serve each request at its die, in index order;
   * an admission to a die with pending refresh quanta first has the die
   * serve the oldest of them (Section D4) */
  for (int64_t i = 0; i < n; i++) {
    int r = orc_classify(m, addr[i]);
    if (r < 0) { in[i] = 0; continue; }
    in[i] = 1;
    orc_loc L = orc_map(m, r, addr[i]);
    if (blocking) {  /* both stages below, per channel */
      key[i] = L.key;
      chan[i] = L.ch;
      n_in++;
      continue;
    }
    int64_t start = db[L.key] ? orc_max(issue[i], df[L.key]) : issue[i];
    if (m->fifo && claimed[L.key] < m->fifo[L.key].len - m->fifo[L.key].head) {
      claimed[L.key]++;
      in[i] = 2;  /* in range, claims a quantum */
      start += tQ;
    }
    dd[i] = start + tR;
    if (dd[i] >= ORC_TIME_LIMIT) overflow = 1;
    df[L.key] = dd[i];
    db[L.key] = 1;
    chan[i] = L.ch;
    ord[n_in].dd = dd[i];
    ord[n_in].idx = i;
    n_in++;
  }
  int nomem = 0;
  if (blocking)
    overflow |= orc_blocking_stage(m, issue, n, in, key, chan, dd, complete, df, db, cf, cb, claimed, tQ, &nomem);
  if (nomem) {
    free(claimed); free(df); free(db); free(cf); free(cb); free(dd); free(chan); free(in); free(ord); free(key);
    return ORC_ENOMEM;
  }
  /* 4. channel service order: by (die_done, index) */
  if (!blocking) qsort(ord, (size_t)n_in, sizeof(orc_pair), orc_cmp_pair);
  /* 5. channel stage */
  for (int64_t k = 0; !blocking && k < n_in; k++) {
    int64_t i = ord[k].idx;
    uint32_t c = chan[i];
    int64_t start = cb[c] ? orc_max(dd[i], cf[c]) : dd[i];
    complete[i] = start + xfer;
    if (complete[i] >= ORC_TIME_LIMIT) overflow = 1;
    cf[c] = complete[i];
    cb[c] = 1;
  }
  /* 6. native path */
  for (int64_t i = 0; i < n; i++)
    if (!in[i]) complete[i] = issue[i];

  int rc = ORC_OK;
  if (overflow) {
    for (int64_t i = 0; i < n; i++) complete[i] = ORC_TIME_ERROR;
    rc = ORC_ERANGE_TIME;
  } else {
    memcpy(m->die_free, df, sizeof(int64_t) * m->n_die_keys);
    memcpy(m->die_busy, db, m->n_die_keys);
    memcpy(m->chan_free, cf, sizeof(int64_t) * p->channels);
    memcpy(m->chan_busy, cb, p->channels);
    /* each claimed quantum, oldest first per die, completes tR before the
     * die-done time of the admission that claimed it */
    for (int64_t i = 0; i < n; i++)
      if (in[i] == 2) {
        orc_fifo *f = &m->fifo[orc_map(m, orc_classify(m, addr[i]), addr[i]).key];
        m->qdone[f->id[f->head++]] = dd[i] - tR;
      }
  }
  free(claimed);
  free(df); free(db); free(cf); free(cb); free(dd); free(chan); free(in); free(ord); free(key);
  return rc;
}

/* ---------------------------------------------------------------- refresh
 * Section D4: refresh read-rewrite pairs enter the same die queues as the
 * application's reads, under ids of their own, and the running program pays
 * for them.  Readings (the paper gives no timing for them):
 *  - one quantum = the read and the rewrite of one device page; it occupies
 *    that page's die queue for tQ = tR + tPROG and no channel time (the
 *    page is rewritten inside its die); tPROG is a model parameter;
 *  - each die queue keeps its pending quanta in submission order; a
 *    quantum's id is its position in the sequence of all submitted quanta;
 *  - an application admission to a die queue with pending quanta claims the
 *    oldest one and the die serves it just before the admission's own read
 *    (die service tQ + tR; the quantum completes tR before the read does);
 *  - pending quanta drain while a die is idle only over a window the caller
 *    names (no application read is issued inside it);
 *  - a failed timing call claims nothing; reset drops pending quanta. */

int orc_refresh_configure(orc_model *m, int64_t t_prog_ns) {
  if (!m || t_prog_ns < 0) return ORC_EINVAL;
  /* the longest die service, tQ + tR, stays within the service bound */
  if (2 * m->p.t_read_ns + t_prog_ns > ORC_SERVICE_LIMIT) return ORC_EINVAL;
  m->t_prog_ns = t_prog_ns;
  return ORC_OK;
}

/* Queue quanta for device pages pages[0..nq) in plan order; their ids are
 * *first_id .. *first_id + nq - 1. */
int orc_refresh_submit(orc_model *m, const uint64_t *pages, int64_t nq, int64_t *first_id) {
  if (!m || nq < 0 || (nq > 0 && !pages)) return ORC_EINVAL;
  if (m->p.flags & ORC_FLAG_VMEM_CURVE) return ORC_EINVAL;  /* no die queues on the vmem route */
  if (!m->fifo) {
    m->fifo = (orc_fifo *)calloc(m->n_die_keys, sizeof(orc_fifo));
    if (!m->fifo) return ORC_ENOMEM;
  }
  if (m->nq + nq > m->qcap) {
    int64_t cap = m->qcap ? m->qcap : 64;
    while (cap < m->nq + nq) cap *= 2;
    int64_t *q = (int64_t *)realloc(m->qdone, sizeof(int64_t) * cap);
    if (!q) return ORC_ENOMEM;
    m->qdone = q;
    m->qcap = cap;
  }
  if (first_id) *first_id = m->nq;
  for (int64_t j = 0; j < nq; j++) {
    orc_fifo *f = &m->fifo[orc_locate(m, pages[j]).key];
    if (f->len == f->cap) {
      int64_t cap = f->cap ? 2 * f->cap : 16;
      int64_t *id = (int64_t *)realloc(f->id, sizeof(int64_t) * cap);
      if (!id) return ORC_ENOMEM;
      f->id = id;
      f->cap = cap;
    }
    f->id[f->len++] = m->nq;
    m->qdone[m->nq++] = ORC_REFRESH_PENDING;
  }
  return ORC_OK;
}

/* Serve pending quanta in idle die time inside [t_from, t_to): each die, in
 * its queue order, starts the next quantum at max(its clock, t_from) (t_from
 * if idle since minus infinity) while that quantum ends by t_to. */
int orc_refresh_drain(orc_model *m, int64_t t_from, int64_t t_to) {
  if (!m || t_from < 0 || t_to < t_from || t_to >= ORC_ISSUE_LIMIT) return ORC_EINVAL;
  if (!m->fifo) return ORC_OK;
  const int64_t tQ = m->p.t_read_ns + m->t_prog_ns;
  for (uint32_t k = 0; k < m->n_die_keys; k++) {
    orc_fifo *f = &m->fifo[k];
    while (f->head < f->len) {
      int64_t start = m->die_busy[k] ? orc_max(m->die_free[k], t_from) : t_from;
      if (start + tQ > t_to) break;
      m->qdone[f->id[f->head++]] = start + tQ;
      m->die_free[k] = start + tQ;
      m->die_busy[k] = 1;
    }
  }
  return ORC_OK;
}

/* Pending quanta per die queue, and completion times of quanta 0..nq-1
 * (ORC_REFRESH_PENDING while not served). */
void orc_refresh_pending(const orc_model *m, int64_t *pend) {
  for (uint32_t k = 0; k < m->n_die_keys; k++) pend[k] = m->fifo ? m->fifo[k].len - m->fifo[k].head : 0;
}
int64_t orc_refresh_count(const orc_model *m) { return m->nq; }
void orc_refresh_done(const orc_model *m, int64_t *done) {
  if (m->nq) memcpy(done, m->qdone, sizeof(int64_t) * m->nq);
}

/* ---------------------------------------------------------------- capacity
 * Sections D5 and D6: a capacity range is served from a bounded frame cache
 * in HBM; an access whose page is not resident faults and reads it from the
 * media; the speculative prefetcher then reads ahead the pages after the
 * faulting one.  Prefetch reads never enter the timing path (D6), so the
 * cache only decides which accesses become media reads.  Readings (the paper
 * names no replacement policy and no prefetch depth):
 *  - pages are numbered within the capacity range, [0, range_pages);
 *  - F frames with FIFO replacement: every insertion takes the frame that
 *    was filled longest ago; a hit changes nothing;
 *  - a fault on page p inserts p, then, for k = 1 .. d in that order while
 *    p + k < range_pages, inserts p + k if it is not resident at that moment
 *    (one prefetch read each);
 *  - a prefetched page counts as used at its first hit and as unused if it
 *    is evicted before one.
 */
typedef struct {
  int64_t frames, degree, range_pages;
  int64_t *frame_page;   /* page held by each frame, -1 = empty */
  uint8_t *frame_pf;     /* 1 = prefetched and not hit since */
  int64_t *slot;         /* frame holding each page, -1 = not resident */
  int64_t head;          /* next frame to fill (the oldest) */
  int64_t hits, misses, pf_reads, pf_used, pf_unused;
} orc_cache;

void orc_cache_destroy(orc_cache *c) {
  if (!c) return;
  free(c->frame_page); free(c->frame_pf); free(c->slot); free(c);
}

void orc_cache_reset(orc_cache *c) {
  for (int64_t f = 0; f < c->frames; f++) { c->frame_page[f] = -1; c->frame_pf[f] = 0; }
  for (int64_t q = 0; q < c->range_pages; q++) c->slot[q] = -1;
  c->head = c->hits = c->misses = c->pf_reads = c->pf_used = c->pf_unused = 0;
}

int orc_cache_create(int64_t frames, int64_t degree, int64_t range_pages, orc_cache **out) {
  if (!out || frames < 1 || degree < 0 || degree >= frames || range_pages < 1) return ORC_EINVAL;
  orc_cache *c = (orc_cache *)calloc(1, sizeof(orc_cache));
  if (!c) return ORC_ENOMEM;
  c->frames = frames; c->degree = degree; c->range_pages = range_pages;
  c->frame_page = (int64_t *)malloc(sizeof(int64_t) * frames);
  c->frame_pf = (uint8_t *)malloc(frames);
  c->slot = (int64_t *)malloc(sizeof(int64_t) * range_pages);
  if (!c->frame_page || !c->frame_pf || !c->slot) { orc_cache_destroy(c); return ORC_ENOMEM; }
  orc_cache_reset(c);
  *out = c;
  return ORC_OK;
}

/* Put page q into the oldest frame; returns nothing, updates the counters. */
static void orc_cache_insert(orc_cache *c, int64_t q, int prefetched) {
  int64_t f = c->head;
  int64_t old = c->frame_page[f];
  if (old >= 0) {
    c->slot[old] = -1;
    if (c->frame_pf[f]) c->pf_unused++;
  }
  c->frame_page[f] = q;
  c->frame_pf[f] = (uint8_t)prefetched;
  c->slot[q] = f;
  c->head = (f + 1) % c->frames;
}

/* Serve pages[0..n) in order.  hit[i] = 1 if access i found its page
 * resident, 0 if it faulted.  The first pf_cap prefetch reads issued, in
 * order, go to pf_page / pf_src (the faulting access); *n_pf = the number
 * issued.  Pages outside the range: EINVAL before anything changes. */
int orc_cache_access(orc_cache *c, const uint64_t *pages, int64_t n, uint8_t *hit, uint64_t *pf_page,
                     int64_t *pf_src, int64_t pf_cap, int64_t *n_pf) {
  if (!c || n < 0 || (n > 0 && (!pages || !hit)) || pf_cap < 0) return ORC_EINVAL;
  for (int64_t i = 0; i < n; i++)
    if (pages[i] >= (uint64_t)c->range_pages) return ORC_EINVAL;
  int64_t npf = 0;
  for (int64_t i = 0; i < n; i++) {
    const int64_t p = (int64_t)pages[i];
    if (c->slot[p] >= 0) {
      hit[i] = 1;
      c->hits++;
      if (c->frame_pf[c->slot[p]]) { c->frame_pf[c->slot[p]] = 0; c->pf_used++; }
      continue;
    }
    hit[i] = 0;
    c->misses++;
    orc_cache_insert(c, p, 0);
    for (int64_t k = 1; k <= c->degree && p + k < c->range_pages; k++) {
      if (c->slot[p + k] >= 0) continue;
      orc_cache_insert(c, p + k, 1);
      c->pf_reads++;
      if (npf < pf_cap && pf_page) { pf_page[npf] = (uint64_t)(p + k); pf_src[npf] = i; }
      npf++;
    }
  }
  if (n_pf) *n_pf = npf;
  return ORC_OK;
}

/* hits, faults, prefetch reads, prefetched pages used, evicted unused. */
void orc_cache_counts(const orc_cache *c, int64_t *out) {
  out[0] = c->hits; out[1] = c->misses; out[2] = c->pf_reads; out[3] = c->pf_used; out[4] = c->pf_unused;
}

void orc_cache_frames(const orc_cache *c, int64_t *frame_page, int64_t *head) {
  memcpy(frame_page, c->frame_page, sizeof(int64_t) * c->frames);
  *head = c->head;
}

/* Die-stage completion times alone (a diagnostic used by the tests): the
 * same step 3 as above, without touching the model's clocks.  Out-of-range
 * requests get ORC_TIME_ERROR. */
int orc_die_done(const orc_model *m, const uint64_t *addr, const int64_t *issue, int64_t n,
                 int64_t *dd) {
  if (!m || n < 0) return ORC_EINVAL;
  int64_t *df = (int64_t *)malloc(sizeof(int64_t) * (m->n_die_keys ? m->n_die_keys : 1));
  uint8_t *db = (uint8_t *)malloc(m->n_die_keys ? m->n_die_keys : 1);
  if (!df || !db) { free(df); free(db); return ORC_ENOMEM; }
  memcpy(df, m->die_free, sizeof(int64_t) * m->n_die_keys);
  memcpy(db, m->die_busy, m->n_die_keys);
  for (int64_t i = 0; i < n; i++) {
    int r = orc_classify(m, addr[i]);
    if (r < 0) { dd[i] = ORC_TIME_ERROR; continue; }
    orc_loc L = orc_map(m, r, addr[i]);
    int64_t start = db[L.key] ? orc_max(issue[i], df[L.key]) : issue[i];
    dd[i] = start + m->p.t_read_ns;
    df[L.key] = dd[i];
    db[L.key] = 1;
  }
  free(df); free(db);
  return ORC_OK;
}

/* Resource clocks, idle encoded as INT64_MIN (for state comparisons). */
void orc_get_state(const orc_model *m, int64_t *die_free, int64_t *chan_free) {
  for (uint32_t k = 0; k < m->n_die_keys; k++) die_free[k] = m->die_busy[k] ? m->die_free[k] : INT64_MIN;
  for (uint32_t c = 0; c < m->p.channels; c++) chan_free[c] = m->chan_busy[c] ? m->chan_free[c] : INT64_MIN;
}

/* Restore resource clocks (checkpoint / resume of an online model).  Idle is
 * INT64_MIN; any other value must lie in [0, 2^62). */
int orc_set_state(orc_model *m, const int64_t *die_free, const int64_t *chan_free) {
  for (uint32_t k = 0; k < m->n_die_keys; k++)
    if (die_free[k] != INT64_MIN && (die_free[k] < 0 || die_free[k] >= ORC_TIME_LIMIT)) return ORC_EINVAL;
  for (uint32_t c = 0; c < m->p.channels; c++)
    if (chan_free[c] != INT64_MIN && (chan_free[c] < 0 || chan_free[c] >= ORC_TIME_LIMIT)) return ORC_EINVAL;
  for (uint32_t k = 0; k < m->n_die_keys; k++) {
    m->die_busy[k] = die_free[k] != INT64_MIN;
    m->die_free[k] = m->die_busy[k] ? die_free[k] : 0;
  }
  for (uint32_t c = 0; c < m->p.channels; c++) {
    m->chan_busy[c] = chan_free[c] != INT64_MIN;
    m->chan_free[c] = m->chan_busy[c] ? chan_free[c] : 0;
  }
  return ORC_OK;
}

/* bf16 -> double, exact: a bf16 is the top 16 bits of an IEEE binary32. */
static double orc_bf16(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Grouped GEMV of the instrumented kernel, in double precision over the exact
 * bf16 inputs:  Y[e][b][nn] = sum_k X[e][b][k] * W[e][nn][k].
 * W is [E][N][K] (each output row's K weights contiguous), X is [E][B][K]. */
int orc_gemv_bf16(const uint16_t *W, int E, int K, int N, const uint16_t *X, int B, double *Y) {
  if (!W || !X || !Y || E <= 0 || K <= 0 || N <= 0 || B <= 0) return ORC_EINVAL;
  for (int e = 0; e < E; e++)
    for (int b = 0; b < B; b++)
      for (int nn = 0; nn < N; nn++) {
        const uint16_t *w = W + ((size_t)e * N + nn) * K;
        const uint16_t *x = X + ((size_t)e * B + b) * K;
        double s = 0.0;
        for (int k = 0; k < K; k++) s += orc_bf16(x[k]) * orc_bf16(w[k]);
        Y[((size_t)e * B + b) * N + nn] = s;
      }
  return ORC_OK;
}
