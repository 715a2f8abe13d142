/*
 * hbf.h -- C ABI of the MI355X (gfx950) HBF service-model hot path.
 *
 * HBFSim (arXiv 2609.09800) models High-Bandwidth Flash as a running GPU
 * program sees it: applications register HBF address ranges, every access is
 * classified against them, and each in-range access is given a modeled
 * completion time by an online media model; the running kernel pays that
 * delay where it first consumes the value.  This library implements that
 * path as batch calls on device arrays:
 *
 *   hbf_register_range   -- explicit ranges (Section "D1: An Explicit and
 *                           Fail-Closed Boundary")
 *   hbf_classify_map     -- classification + page-geometry mapping (D1)
 *   hbf_time_requests    -- modeled completion of every request (Section
 *                           "Design": each foreground request enters the
 *                           online media model and its completion returns to
 *                           that request)
 *   hbf_gemv_instrumented-- a bf16 grouped GEMV whose weight pages wait for
 *                           their modeled completion at the point of
 *                           consumption (Section "D2: Preserving GPU
 *                           Asynchrony")
 *
 * Timing model.  The paper leaves the media model to MQSim and publishes no
 * HBF timing parameters, so this library fixes one reading and documents
 * it: each request is a one-page read that first occupies its die for
 * t_read_ns (FCFS by (issue time, request index)) and then its channel for
 * xfer_ns = ceil(page_bytes * 1e9 / channel_bytes_per_s) (FCFS by (die-done
 * time, request index)).  Buffers between the stages are unbounded.  Pages
 * are striped channel-first: for device page p, ch = p mod C,
 * die = (p / C) mod D, plane = (p / (C*D)) mod P, page = p / (C*D*P).
 * Device pages number the registered ranges in registration order.  The die
 * queue is (ch, die), or (ch, die, plane) with HBF_FLAG_PLANE_PARALLEL.
 * All times are int64 nanoseconds; results are exact integers.
 *
 * Conventions for every call:
 *  - Pointers named dev_* / device arrays live in GPU memory of the current
 *    HIP device; host_* pointers are host memory.  The caller owns every
 *    array it passes; the library never frees caller memory.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls that
 *    launch work are asynchronous on that stream and return once enqueued.
 *  - Host-detectable errors return a negative code before any launch and
 *    leave every output untouched.
 *  - Device-detected errors (bad issue times, time-domain overflow) are
 *    fail-closed: every complete_ns[i] of that call is written as
 *    HBF_TIME_ERROR before the error is recorded, resource clocks keep their
 *    values from before the call, and hbf_get_status() reports the error.
 *  - A model handle is not thread-safe; calls on one handle must be ordered
 *    on one stream (or externally synchronised).
 */
#ifndef HBF_H_
#define HBF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define HBF_OK             0
#define HBF_EINVAL        -1  /* invalid argument or parameter */
#define HBF_EALIGN        -2  /* range not page aligned / not a page multiple */
#define HBF_EOVERLAP      -3  /* range overlaps a registered range */
#define HBF_ENOWORKSPACE  -4  /* caller workspace smaller than hbf_workspace_bytes */
#define HBF_EUNSORTED     -5  /* issue_ns decreases somewhere (device-detected) */
#define HBF_ERANGE_TIME   -6  /* issue_ns outside [0, 2^61) or a modeled time
                                 reached 2^62 (device-detected) */
#define HBF_EHIP          -7  /* a HIP runtime call failed */
#define HBF_ENOMEM        -8  /* host or device allocation failed */
#define HBF_EINTERNAL     -9  /* a bounded device-side wait ran out (an internal
                                 fault: the call failed closed) */

/* complete_ns value written for every request of a failed call. */
#define HBF_TIME_ERROR    INT64_MIN

/* hbf_params.flags */
#define HBF_FLAG_PLANE_PARALLEL 1u  /* die queues keyed by (ch, die, plane) */
/* Media variant: die page-register blocking.  Each die queue holds one page
 * register: a read leaves its page there, and the die starts no other read
 * until that page's channel transfer has completed (the page has left the
 * register).  Channels still serve pages FCFS by (die-done, index).  The
 * die's clock after a call is its last transfer's completion.  Timed per
 * channel in service order (one wave per channel): slower than the default
 * unblocked model, which needs no such order. */
#define HBF_FLAG_REGISTER_BLOCKING 2u
/* Timing source: the calibrated end-to-end vmem curve (Section
 * "Discussion") instead of the media model.  That curve was measured on a
 * host paging path presenting an SSD as memory; it prices a sequential
 * burst of L pages, T(L), from knots at 1, 4, 16, 64, 256 and 512 pages
 * (hbf_vmem_configure).  Reading used here: between knots T is linear in L,
 * rounded down to whole ns; past 512 pages T(L) = T(512) +
 * floor((T(512) - T(256)) * (L - 512) / 256).  An in-range access continues
 * the burst iff its device page is the one after the previous in-range
 * access's page (request order, across calls until reset); any other access
 * (a jump, a step back, the same page again) starts a burst of one.  The
 * route serves one access at a time in request order, the access at burst
 * position L taking T(L) - T(L-1):
 *   complete = max(issue, route free) + T(L) - T(L-1).
 * Out-of-range requests take the native path (complete = issue).  No die or
 * channel queues: refresh calls return HBF_EINVAL; not combinable with
 * HBF_FLAG_REGISTER_BLOCKING (HBF_EINVAL at create).  The route's clock and
 * burst persist across calls and are cleared by hbf_model_reset;
 * hbf_get_state / hbf_set_state cover the media clocks only. */
#define HBF_FLAG_VMEM_CURVE 4u

typedef struct hbf_model *hbf_model_t;  /* opaque, owned by the library */

/* Device geometry and timing.  All integers: there is no floating point on
 * the timing path. */
typedef struct {
  uint32_t channels;          /* C, 1..1024 */
  uint32_t dies_per_channel;  /* D, 1..256 */
  uint32_t planes_per_die;    /* P, 1..64 */
  uint32_t page_bytes;        /* bytes per page (one request reads one page) */
  int64_t  t_read_ns;         /* tR, die read time, 1..2^29 */
  uint64_t channel_bytes_per_s; /* channel bandwidth in bytes/s (decimal GB) */
  uint32_t flags;             /* HBF_FLAG_* */
} hbf_params;

/* Create a model.  Validates `params` entirely on the host (C*D*P <= 65536,
 * die queues per channel <= 64, die queues <= 2048, xfer_ns in 1..2^29) and
 * returns HBF_EINVAL
 * without touching the GPU if they are invalid.  Resource clocks start
 * "idle since minus infinity".  Device state is allocated on the current
 * HIP device at the first call that needs it.  *out receives the handle. */
int hbf_model_create(const hbf_params *params, hbf_model_t *out);

/* Release the model and everything the library allocated for it.  Waits for
 * the model's outstanding work. NULL is ignored. */
void hbf_model_destroy(hbf_model_t model);

/* Derived channel transfer time per page, in ns (host query, no GPU). */
int hbf_xfer_ns(hbf_model_t model, int64_t *xfer_ns);

/* Number of die queues: C*D, or C*D*P with HBF_FLAG_PLANE_PARALLEL. */
int hbf_n_die_queues(hbf_model_t model, uint32_t *n);

/* Return every resource clock to "idle since minus infinity" (enqueued on
 * `stream`). */
int hbf_model_reset(hbf_model_t model, void *stream);

/* Register the address interval [base, base+bytes) as an HBF range
 * (Section D1).  base and bytes must be multiples of page_bytes
 * (HBF_EALIGN), bytes > 0, the interval must not wrap 2^64 (HBF_EINVAL) and
 * must not overlap a registered range (HBF_EOVERLAP).  At most 64 ranges.
 * The range's device pages follow those of earlier-registered ranges.
 * Registration takes effect for calls made after it returns (the device
 * sees an immutable snapshot per call).  Host only; *range_id (nullable)
 * receives the registration index. */
int hbf_register_range(hbf_model_t model, uint64_t base, uint64_t bytes, int32_t *range_id);

/* Device scratch needed by hbf_time_requests for n requests, in bytes. */
int hbf_workspace_bytes(hbf_model_t model, int64_t n, size_t *bytes);

/* Use caller-owned device memory dev_ptr[0..bytes) as scratch (it must stay
 * valid while calls that use it run; pass NULL, 0 to go back to
 * library-owned scratch, which the library allocates and grows itself).
 * A later hbf_time_requests whose need exceeds `bytes` returns
 * HBF_ENOWORKSPACE. */
int hbf_set_workspace(hbf_model_t model, void *dev_ptr, size_t bytes);

/* Classification and page mapping of n addresses (Section D1).
 * dev_addr: uint64[n] byte addresses (device).  dev_map_out: uint64[n]
 * (device), one packed word per address:
 *   bit 63      1 = inside a registered range, 0 = native path (word is 0)
 *   bits 62..56 range index (registration order)
 *   bits 55..50 plane, bits 49..42 die, bits 41..32 channel
 *   bits 31..0  page index within the plane
 * Requires C <= 1024, D <= 256, P <= 64 and page index < 2^32 (HBF_EINVAL
 * if a page index overflows: detected on the device, reported by
 * hbf_get_status, that element's word is 0).  n may be 0. */
int hbf_classify_map(hbf_model_t model, const uint64_t *dev_addr, int64_t n, uint64_t *dev_map_out,
                     void *stream);

/* Modeled completion time of n page-read requests.
 * dev_addr: uint64[n] byte addresses; dev_issue_ns: int64[n] issue times,
 * nondecreasing in index, each in [0, 2^61); dev_complete_ns: int64[n]
 * output (all device memory, 0 <= n <= 2^31).  In-range requests get the
 * completion of the die-read + channel-transfer model above; requests
 * outside every range get complete = issue (native path, no modeled delay).
 * Resource clocks persist across calls and a call is a barrier: every
 * request of a call is served at its die and channel before any request of
 * a later call.  Device-detected errors: HBF_EUNSORTED, HBF_ERANGE_TIME
 * (fail-closed, see above).  Returns HBF_OK once enqueued. */
int hbf_time_requests(hbf_model_t model, const uint64_t *dev_addr, const int64_t *dev_issue_ns,
                      int64_t n, int64_t *dev_complete_ns, void *stream);

/* ---- The same call without any allocation, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid device allocation).  Arguments, results, device-detected
 * errors and the model's clocks are those of hbf_time_requests; the call
 * allocates nothing (no hipMalloc / hipFree, no workspace of the model, no
 * profiling events).  Its scratch is one static device array of
 * HBF_NOALLOC_SCRATCH_BYTES per GPU, held from the first such call on that
 * GPU until the process ends and shared by every such call on it: calls
 * that overlap on one GPU (other streams, other models) race on it and must
 * be ordered by the caller.  Host-detected errors, before any launch:
 * HBF_EINVAL for the arguments hbf_time_requests refuses, or if the
 * model's device state does not exist yet on the current HIP device (any
 * earlier call that launches work creates it, e.g. hbf_model_reset);
 * HBF_ENOWORKSPACE if hbf_workspace_bytes(model, n) exceeds
 * HBF_NOALLOC_SCRATCH_BYTES (up to about 4 M requests on the 16 x 8 x 4
 * geometry, 2.9 M with 2,048 die queues). */
#define HBF_NOALLOC_SCRATCH_BYTES (64ull << 20)
int hbf_time_requests_noalloc(hbf_model_t model, const uint64_t *dev_addr, const int64_t *dev_issue_ns,
                              int64_t n, int64_t *dev_complete_ns, void *stream);

/* Closed-loop timing of a layered decode: the running program pays each
 * layer's modeled delays before it issues the next layer's reads (Section
 * "Introduction": delays are paid by the running program; Section D2: the
 * wait sits where the loaded values are first used, here the next layer).
 * The n requests form L consecutive layers: layer l is
 * [host_layer_start[l], host_layer_start[l+1]) (host array of L+1 entries,
 * nondecreasing, first 0, last n; empty layers allowed).  Every request of
 * layer l is issued at
 *     t_0 = t_start_ns,   t_(l+1) = done_l + compute_ns,
 *     done_l = max(t_l, max over layer l of complete_ns)
 * and is timed on the persistent model exactly as one hbf_time_requests call
 * holding that layer would time it.  All on `stream`; no host round trip.
 * Outputs (device): dev_issue_ns[n] (the issue times assigned),
 * dev_complete_ns[n], dev_layer_done_ns[L].  t_start_ns and compute_ns in
 * [0, 2^61).  Device-detected errors fail the layer as in hbf_time_requests;
 * its done time becomes HBF_TIME_ERROR and every later layer fails too. */
int hbf_time_layers(hbf_model_t model, const uint64_t *dev_addr, int64_t n,
                    const int64_t *host_layer_start, int L, int64_t t_start_ns, int64_t compute_ns,
                    int64_t *dev_issue_ns, int64_t *dev_complete_ns, int64_t *dev_layer_done_ns,
                    void *stream);

/* Instrumented grouped GEMV with delay injection at consumption
 * (Section D2: issue is split from consumption; the wait sits at the first
 * use of the loaded value).
 *   Y[e][b][nn] = sum_k X[e][b][k] * W[e][nn][k]   (fp32 accumulate)
 * dev_W: bf16 bits [E][N][K] (each output row's K weights contiguous),
 *   lying inside one registered range, page aligned;  dev_X: bf16 bits
 *   [E][B][K] (16-byte aligned);  dev_Y: float [E][B][N].  K must be a
 *   multiple of 512, at most 4096, with 2*K dividing page_bytes, at most
 *   16 rows per page, and N a multiple of the rows per page.
 * dev_page_issue_ns / dev_page_complete_ns: int64 per weight page
 *   (E*N*K*2 / page_bytes entries, page order of W), e.g. from
 *   hbf_time_requests.  Every page of the call is issued at the call's
 *   start: its time origin is the GPU wall clock (constant rate, see
 *   hbf_wall_clock_tick_ps) at which the consuming kernel's first workgroup began.
 *   Page q's loads are issued before its first use, and that use waits
 *   until origin + (complete[q] - issue[q]) ns.  The call runs on at most
 *   as many workgroups as the GPU holds at once, each taking its pages in
 *   ascending order of delay, so no page waits behind another page's delay.
 *   Both NULL: no delay (one workgroup per page, no clock reads).  Times
 *   outside [0, 2^62) or complete[q] < issue[q]: no wait for that page and
 *   HBF_ERANGE_TIME from hbf_get_status; a delay above 1 s is clamped to
 *   1 s and reported the same way (the GPU never spins longer).
 * dev_measured_delay_ns (nullable, needs the time arrays): int64 per page,
 *   the time from the call's origin to the page's release (wall-clock
 *   ticks * tick length), for injection-fidelity checks.  Calls with delays
 *   on one model must not overlap (they share the origin record).
 * 1 <= B <= 64, E >= 1. */
int hbf_gemv_instrumented(hbf_model_t model, const uint16_t *dev_W, int E, int K, int N,
                          const uint16_t *dev_X, int B, float *dev_Y,
                          const int64_t *dev_page_issue_ns, const int64_t *dev_page_complete_ns,
                          int64_t *dev_measured_delay_ns, void *stream);

/* Knot values of the vmem curve (model created with HBF_FLAG_VMEM_CURVE):
 * host_knot_ns[6] = T(1), T(4), T(16), T(64), T(256), T(512) in ns.  The
 * paper prints T(1) = 11,133 ns and none of the others; until configured a
 * model uses T(L) = 11,133 * L at every knot (no burst benefit).  Requires
 * 1 <= T(1) <= 2^29, nondecreasing knots, and at most 2^29 ns per page on
 * average over every segment (else HBF_EINVAL).  Host only; applies to
 * calls made after it returns. */
int hbf_vmem_configure(hbf_model_t model, const int64_t *host_knot_ns);

/* ---- Refresh traffic in the same queues (Section "D4: Retention, Refresh,
 * and Wear as Injected Latency": refresh read-rewrite pairs get ids of their
 * own, enter the same queues as the application's reads, and one
 * admission can take a single refresh quantum along, served ahead of it).
 * Reading used here (the paper gives no refresh timing):
 *  - one quantum = the read and the rewrite of one device page; it occupies
 *    that page's die queue for tQ = t_read_ns + t_prog_ns and no channel
 *    time (the page is rewritten inside its die);
 *  - each die queue holds its pending quanta in submission order; every
 *    in-range admission to a die queue with quanta pending claims the
 *    oldest one: the die serves it right before the admission's read, so
 *    that read's die service is tQ + t_read_ns and the quantum completes
 *    t_read_ns before the read leaves the die;
 *  - pending quanta drain in idle die time only over a window the caller
 *    names (hbf_refresh_drain);
 *  - a call that fails (device-detected error) claims nothing; reset drops
 *    every pending quantum.
 * With quanta pending, hbf_time_requests / hbf_time_layers run one extra
 * counting pass over the addresses. */

/* One eligible erase block of a refresh plan. */
typedef struct {
  uint32_t epoch;    /* eligibility epoch */
  uint32_t zone;
  uint32_t channel, die, plane;
  uint32_t block;    /* block index within its plane */
} hbf_refresh_block;

/* Device pages of a refresh plan in the scheduler's deterministic order
 * (Section D4: eligibility epoch, then channel round robin, then die round
 * robin, then zone, block and page).  Host-only, no model needed.
 * Block b of plane (channel, die, plane) holds that plane's pages
 * b*pages_per_block .. (b+1)*pages_per_block - 1; plane page pg is device
 * page ((pg*P + plane)*D + die)*C + channel.  Within an epoch, rounds visit
 * the channels that still have pages in ascending order, and each visit
 * takes one page from the channel's next die (cyclically after the die it
 * served last, lowest first) that still has pages; a die's pages go in
 * (zone, block, plane, page) order.  host_pages_out receives
 * n_blocks * pages_per_block entries (capacity `cap`, else HBF_EINVAL).
 * Block fields out of the geometry: HBF_EINVAL.  A physical block
 * (channel, die, plane, block) is eligible at most once per epoch, so a
 * plan listing one twice in an epoch (under any zone) is refused with
 * HBF_EINVAL; in different epochs it is refreshed once per epoch. */
int hbf_refresh_plan(const hbf_params *params, const hbf_refresh_block *host_blocks, int64_t n_blocks,
                     uint32_t pages_per_block, uint64_t *host_pages_out, int64_t cap);

/* Set tPROG, the page program time of a refresh rewrite (>= 0, with
 * 2 * t_read_ns + t_prog_ns <= 2^29).  Required before hbf_refresh_submit;
 * applies to quanta served from the next call on. */
int hbf_refresh_configure(hbf_model_t model, int64_t t_prog_ns);

/* Queue one quantum per device page host_pages[0..nq), in that (plan)
 * order.  dev_done_ns: int64[nq] device array that receives quantum j's
 * completion time when it is served (claimed by an admission or drained);
 * the library fills it with -1 (pending) now.  The caller keeps it alive
 * while any of its quanta is pending (until reset, or until
 * hbf_refresh_pending reports none).  Synchronises `stream` (the host
 * rebuilds the pending lists).  0 <= nq <= 2^31. */
int hbf_refresh_submit(hbf_model_t model, const uint64_t *host_pages, int64_t nq, int64_t *dev_done_ns,
                       void *stream);

/* Serve pending quanta in idle die time inside [t_from_ns, t_to_ns): each
 * die queue, oldest quantum first, starts the next one at max(its clock,
 * t_from_ns) while it ends by t_to_ns, and its clock advances.  The caller
 * promises no admission is issued inside the window.
 * 0 <= t_from_ns <= t_to_ns < 2^61.  Asynchronous on `stream`. */
int hbf_refresh_drain(hbf_model_t model, int64_t t_from_ns, int64_t t_to_ns, void *stream);

/* Pending quanta per die queue (host_pending[n_die_queues]), after
 * synchronising `stream`. */
int hbf_refresh_pending(hbf_model_t model, uint32_t *host_pending, void *stream);

/* ---- Capacity mode: frame cache and next-page prefetcher (Section "D5:
 * Capacity": a capacity range is served from a bounded frame cache in HBM,
 * a miss reads the page from the media; Section "D6: Speculative
 * Prefetcher": once a fault is served, the next pages are read ahead,
 * and prefetch reads never enter the timing path).  This step decides which
 * accesses become media reads; a faulting access is then timed like any
 * other read (e.g. by hbf_time_requests on the faulting accesses).
 * Reading used here (the paper names no replacement policy or depth):
 *  - pages are numbered within the capacity range, [0, range_pages);
 *  - `frames` frames, FIFO replacement: every insertion takes the frame
 *    filled longest ago, a hit changes nothing;
 *  - a fault on page p inserts p, then for k = 1 .. prefetch_pages in that
 *    order while p + k < range_pages, inserts p + k if it is not resident
 *    at that moment (one prefetch read each);
 *  - a prefetched page counts as used at its first hit and as unused if it
 *    is evicted before one.
 * 1 <= frames < 2^31, prefetch_pages < frames and <= 63,
 * 1 <= range_pages <= 2^31.  The cache state lives on the current HIP
 * device and persists across calls until reset. */
typedef struct hbf_cache *hbf_cache_t;  /* opaque, owned by the library */

/* Create an empty cache (allocates frames*12 bytes of device memory for up
 * to 63 frames, range_pages*8 + frames*2 bytes above; caches of 64 frames
 * or more over at most 2^26 range pages also hold the chunk state below,
 * range_pages*24 bytes and about 3.1 MiB;
 * synchronous). */
int hbf_cache_create(uint32_t frames, uint32_t prefetch_pages, uint64_t range_pages, hbf_cache_t *out);
void hbf_cache_destroy(hbf_cache_t cache);
/* Empty every frame and zero the counters (asynchronous on `stream`). */
int hbf_cache_reset(hbf_cache_t cache, void *stream);

/* Serve dev_pages[0..n) (uint64 page numbers within the range) in order.
 * dev_hit[n] (uint8): 1 = the page was resident, 0 = the access faulted.
 * dev_pf_page / dev_pf_src (both NULL or both set): the first pf_cap
 * prefetch reads issued by this call, in order: page, and the index of the
 * faulting access that issued it.  dev_counts (int64[8], device): [0..4]
 * hits, faults, prefetch reads, prefetched pages used, prefetched pages
 * evicted unused, all since the last reset; [5] prefetch reads issued by
 * this call; [6] 0, or HBF_EINVAL if some page was >= range_pages (then
 * nothing changed and dev_hit is not written); [7] 0.  Asynchronous. */
int hbf_cache_access(hbf_cache_t cache, const uint64_t *dev_pages, int64_t n, uint8_t *dev_hit,
                     uint64_t *dev_pf_page, int64_t *dev_pf_src, int64_t pf_cap, int64_t *dev_counts,
                     void *stream);

/* Accesses served together (default: frames/16 clamped to [16384, 262144]
 * for caches with chunk state, else 0).  A call is
 * cut into chunks of that many accesses.  Each chunk is first solved in
 * parallel as if nothing were evicted: an access faults only as the first
 * access of a page not resident when the chunk began, unless an earlier
 * fault at most prefetch_pages below it inserted the page.  That answer
 * is kept only if every hit and every prefetch candidate it found resident
 * is still within the last `frames` insertions at that moment, which makes
 * it exactly the FIFO answer.  Otherwise the chunk is served one access
 * after another.  The results do not depend on the chunk length.
 * 0 <= accesses <= 262144; a nonzero value needs chunk state (HBF_EINVAL
 * otherwise).  Host only. */
int hbf_cache_set_chunk(hbf_cache_t cache, uint32_t accesses);
int hbf_cache_get_chunk(hbf_cache_t cache, uint32_t *accesses);

/* Many caches over one stream at once (a sweep of frame budgets and
 * prefetch depths): configuration b has host_frames[b] frames and
 * host_prefetch[b] prefetch pages, starts empty, and serves all of
 * dev_pages[0..n).  dev_counts: int64[n_cfg][5], the five counters of
 * each.  1 <= n_cfg <= 65535.  Caches that have a default chunk length
 * (see hbf_cache_set_chunk) are served chunk by chunk with the smallest of
 * those lengths.  Allocates the caches' state for the call (about
 * range_pages*32 bytes per cache of 64 frames or more over at most 2^26
 * range pages, range_pages*8 for larger ranges, frames*12 below 64 frames;
 * HBF_ENOMEM if that does not fit) and synchronises `stream` before
 * returning; returns HBF_EINVAL if some page was >= range_pages (counts
 * then all zero). */
int hbf_cache_sweep(const uint32_t *host_frames, const uint32_t *host_prefetch, int n_cfg, uint64_t range_pages,
                    const uint64_t *dev_pages, int64_t n, int64_t *dev_counts, void *stream);

/* Wall-clock tick of the delay injection, in picoseconds (10,000 for a
 * 100 MHz counter).  Needs the GPU. */
int hbf_wall_clock_tick_ps(hbf_model_t model, int64_t *tick_ps);

/* Synchronise `stream`, then return and clear the sticky device status:
 * HBF_OK, HBF_ERANGE_TIME, HBF_EUNSORTED, HBF_EINVAL or HBF_EINTERNAL (in
 * that order of precedence); HBF_EHIP if synchronising or reading the
 * status fails. */
int hbf_get_status(hbf_model_t model, void *stream);

/* Copy the resource clocks to host memory after synchronising `stream`:
 * host_die_free[n_die_queues], host_chan_free[channels]; an idle clock
 * reads INT64_MIN.  Either pointer may be NULL. */
int hbf_get_state(hbf_model_t model, int64_t *host_die_free, int64_t *host_chan_free, void *stream);

/* Restore clocks saved by hbf_get_state (checkpoint / resume).  Each value
 * is INT64_MIN (idle) or in [0, 2^62), else HBF_EINVAL.  Synchronous. */
int hbf_set_state(hbf_model_t model, const int64_t *host_die_free, const int64_t *host_chan_free,
                  void *stream);

/* Per-kernel timing of hbf_time_requests (diagnostics).  hbf_profile(m, 1)
 * starts a new record: every later call records HIP events between its
 * kernels on its own stream (the last 64 calls are kept).  hbf_kernel_times
 * synchronises on the last recorded call and returns, in launch order, each
 * kernel's name and its mean duration (ms) over the recorded calls. */
int hbf_profile(hbf_model_t model, int enable);
int hbf_kernel_times(hbf_model_t model, float *host_ms, const char **host_names, int max, int *count);

/* Static string for a status code. */
const char *hbf_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* HBF_H_ */
