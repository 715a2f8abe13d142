// Internal declarations shared by the HIP kernels and the C ABI host code.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "hbf.h"

namespace hbf {

// "Idle since minus infinity".  Every modeled time of a call lies in
// [0, 2^62); the prefix maxima of the Lindley form (time - rank * service)
// stay above -2^60, so -2^61 is below every value that can occur.
constexpr int64_t NEG = -(int64_t(1) << 61);
constexpr int64_t ISSUE_LIMIT = int64_t(1) << 61;
constexpr int64_t TIME_LIMIT = int64_t(1) << 62;
constexpr int64_t SERVICE_LIMIT = int64_t(1) << 29;
constexpr int64_t N_LIMIT = int64_t(1) << 31;
constexpr int MAX_RANGES = 64;
constexpr int MAX_KEYS = 2048;      // die queues
constexpr int MAX_CHANNELS = 1024;
constexpr uint16_t KEY_NONE = 0xFFFF;

// per-call / sticky device error bits
constexpr uint32_t ERR_RANGE_TIME = 1u;
constexpr uint32_t ERR_UNSORTED = 2u;
constexpr uint32_t ERR_OVERFLOW = 4u;
constexpr uint32_t ERR_MAP = 8u;
constexpr uint32_t ERR_INTERNAL = 16u;  // a bounded internal wait ran out (never expected)

// Die stage: 256 threads (4 wave64), 16 items per thread per chunk.
constexpr int BLK = 256;            // threads per block of the small kernels
constexpr int WAVES = BLK / 64;
constexpr int DBLK = 512;           // threads per block of the two die-stage passes
constexpr int DWAVES = DBLK / 64;
constexpr int DITEMS = 8;           // requests per thread per chunk
constexpr int CHUNK = DBLK * DITEMS;  // 4096 requests staged per chunk
constexpr int TARGET_TILES = 512;   // die-stage tiles: two 512-thread blocks per CU

// Channel stage: a time cell of one channel is merged in LDS if it holds at
// most MCAP requests, otherwise streamed in MCAP-sized rounds.
constexpr int MCAP = 1024;
// Time buckets of width 2^floor(log2 tR) hold at most one request per die;
// a cell of at most 64 such buckets is ranked with per-die bucket masks.
constexpr int MAX_BUCKETS = 64;
// The channel stage hands each XCD (L2 domain) its own time windows, so the
// requests of one window, from every channel, complete in one L2.
constexpr int NXCD = 8;
constexpr int MAX_RUNS = 64;        // die queues per channel (D, or D*P)
// Closed-loop layers in one launch: one workgroup per layer ranks each
// layer's requests, so layers are bounded; larger ones take a call per layer.
constexpr int64_t LAYERS_MAX_LAYER = int64_t(1) << 22;
constexpr int LAYERS_MAX_COUNT = 1 << 20;

// Snapshot of the registered ranges, sorted by base (passed by value).
struct RangeTable {
  uint64_t base[MAX_RANGES];
  uint64_t bytes[MAX_RANGES];
  uint64_t pbase[MAX_RANGES];     // first device page of the range
  uint32_t rid[MAX_RANGES];       // registration index
  int32_t n;
};

// Geometry and timing (passed by value).
struct Geo {
  uint32_t C, D, P;
  uint32_t Dk;        // die queues per channel (D, or D*P)
  uint32_t K;         // die queues (C * Dk)
  uint32_t page_bytes;
  uint32_t plane_parallel;
  uint32_t pow2;      // page_bytes, C, D, P all powers of two
  uint32_t lg_page, lg_C, lg_D, lg_P;
  uint32_t lg_tR;     // floor(log2(tR)): bucket width of the channel merge
  int64_t tR, xfer;
  int64_t tQ;         // die time of one refresh quantum (tR + tPROG), 0 if unset
  uint32_t reg_block; // media variant: die page-register blocking
  uint32_t vmem;      // timing source: the calibrated end-to-end vmem curve
  int64_t vknot[6];   // vmem burst cost T(L) at L = 1, 4, 16, 64, 256, 512 pages
};

// Persistent device state of a model.  Refresh quanta pending at die queue
// k are entries ref_off[k] + ref_head[k] .. + ref_pend[k] - 1 of ref_slot,
// oldest first; each entry points at the caller's cell that receives the
// quantum's completion time.
struct DevState {
  int64_t die_free[MAX_KEYS];     // NEG = idle
  int64_t chan_free[MAX_CHANNELS];
  uint32_t sticky;                // sticky error bits
  uint32_t pad;
  uint32_t ref_pend[MAX_KEYS];
  uint32_t ref_head[MAX_KEYS];
  uint32_t ref_off[MAX_KEYS];
  int64_t **ref_slot;
  // Instrumented GEMV with delays: the time origin of the current call
  // (wall-clock ticks, read by the call's first kernel).
  uint64_t gemv_origin;
  // vmem route: its clock (NEG = idle), the device page of the last
  // in-range access and the length of the burst it ended (vhave = 0: none)
  int64_t vfree;
  uint64_t vlast;
  int64_t vburst;
  uint32_t vhave;
  uint32_t vpad;
};

// Completion cell of a refresh quantum that has not been served.
constexpr int64_t REFRESH_PENDING = -1;

// Per-call control block (in the workspace).
struct CallCtl {
  uint32_t err;       // per-call error bits
  uint32_t n_in;      // in-range requests
  uint32_t G;         // time cells per channel
  uint32_t shift;     // log2(cell width in ns)
  int64_t max_dd;     // largest die-done time of the call
  int64_t max_cpl;    // largest in-range completion of the call (NEG if none)
  int64_t cbase;      // origin of the cell grid (= first issue time)
  uint32_t n_rest;    // cells k_cell_agg lists for k_cell_rest (grids off the bucket path)
  uint32_t wctr;      // next unit of the fused channel stage
};

// Workspace layout of one hbf_time_requests call.
struct Layout {
  int64_t n;
  uint32_t nt;            // die-stage tiles
  int64_t tile_elems;
  uint32_t gmax;          // cell budget per channel
  uint32_t s0;            // minimum cell shift
  size_t off_ctl, off_agg_cnt, off_agg_A, off_tin_L, off_tin_base;
  size_t off_totals, off_seg, off_dfnew, off_cfnew;
  size_t off_dd, off_ix, off_kr, off_lb;
  size_t off_cagg, off_cgin;  // per (channel, time cell): aggregate, entering term
  size_t off_wst;             // fused channel stage: published aggregate and inclusive term per cell
  size_t off_nbl;             // cells k_cell_agg lists for k_cell_rest
  size_t off_iss;             // register blocking: issue times in die order (n int64)
  // vmem route (tiles of VM_TILE requests): per tile its burst summary, the
  // summary of everything before it, its route-clock pair and entering
  // clock; per request its service (u32); the call's closing state
  size_t off_vsum, off_vin, off_vpair, off_vfin, off_vcost, off_vend;
  size_t off_vwsum, off_vwpair;  // the same summary and pair per wave span of a tile
  size_t total;
};

Layout make_layout(const Geo &g, int64_t n);

// Launchers (hbf_kernels.hip).  All enqueue on `s` and return the first
// launch error.
// refresh: quanta may be pending (the die stage then charges them to the
// admissions that claim them; a count pass comes first)
hipError_t launch_time_requests(const Geo &g, const RangeTable &rt, const Layout &L, char *ws,
                                DevState *st, const uint64_t *addr, const int64_t *issue,
                                int64_t *complete, hipStream_t s, hipEvent_t *ev, int n_ev,
                                bool refresh);
// Register-blocking channel stage (hbf_blocking.hip): one wave per channel.
hipError_t launch_regblock(const Geo &g, const uint64_t *DDw, const uint32_t *IX, const int64_t *issue_do,
                           const uint32_t *seg_start, const uint32_t *totals, DevState *st, CallCtl *ctl,
                           int64_t *complete, int64_t *dfnew, int64_t *cfnew, bool ref, hipStream_t s);
// Calibrated vmem curve (hbf_vmem.hip): the whole timing call on the vmem
// route (classification, burst lengths, route clock, complete[]).
constexpr int VM_THREADS = 256;
constexpr int VM_ITEMS = 16;
constexpr int64_t VM_TILE = VM_THREADS * VM_ITEMS;
hipError_t launch_vmem(const Geo &g, const RangeTable &rt, const Layout &L, char *ws, DevState *st,
                       const uint64_t *addr, const int64_t *issue, int64_t *complete, hipStream_t s);
// Closed-loop layers in one launch (hbf_layers.hip): whether a geometry can
// take it on this GPU (every channel's workgroup resident at once), its
// scratch for n requests in L layers, and the launch (host_ls: L + 1 layer
// starts on the host).
bool layers_fast_ok(const Geo &g, int ncu);
size_t layers_ws_bytes(const Geo &g, int64_t n, int L);
hipError_t launch_layers(const Geo &g, const RangeTable &rt, char *ws, DevState *st, const uint64_t *addr,
                         int64_t n, const int64_t *host_ls, int L, int64_t t_start, int64_t compute_ns,
                         int64_t *issue, int64_t *complete, int64_t *done, std::vector<unsigned char> &up,
                         hipEvent_t up_done, hipStream_t s);
hipError_t launch_refresh_drain(const Geo &g, DevState *st, int64_t t_from, int64_t t_to, hipStream_t s);
hipError_t launch_fill(int64_t *p, int64_t n, int64_t v, hipStream_t s);
// Device address of this GPU's static scratch of hbf_time_requests_noalloc
// (HBF_NOALLOC_SCRATCH_BYTES); `dev` must be the current device.
hipError_t noalloc_scratch(int dev, char **ptr);
// Small calls (hbf_small.hip): a whole timing call of at most CHUNK
// requests by one workgroup, for the plain two-stage model with at most
// SMALL_K die queues, at most SMALL_DK per channel.
constexpr uint32_t SMALL_K = 512;
constexpr uint32_t SMALL_DK = 16;
constexpr int SMALL_LDS_MAX = 156 * 1024;  // dynamic LDS; the kernel's static LDS fits beside it in 160 KB
bool small_path_ok(const Geo &g, int64_t n, bool refresh);
hipError_t launch_small(const Geo &g, const RangeTable &rt, DevState *st, CallCtl *ctl, const uint64_t *addr,
                        const int64_t *issue, int64_t n, int64_t *complete, hipStream_t s);
hipError_t set_lds_small();
hipError_t launch_classify(const Geo &g, const RangeTable &rt, DevState *st, const uint64_t *addr,
                           int64_t n, uint64_t *map, hipStream_t s);
hipError_t launch_reset(DevState *st, hipStream_t s);
// Closed-loop layers: write the issue times of one layer / reduce its done time.
hipError_t launch_layer_issue(int64_t *issue, int64_t count, const int64_t *prev_done, int64_t t_start,
                              int64_t compute_ns, hipStream_t s);
hipError_t launch_layer_done(const CallCtl *ctl, int64_t count, const int64_t *prev_done, int64_t t_start,
                             int64_t compute_ns, int64_t *done, hipStream_t s);
hipError_t launch_gemv(const uint16_t *W, int E, int K, int N, int page_bytes, const uint16_t *X,
                       int B, float *Y, const int64_t *pi, const int64_t *pc, int64_t *meas,
                       int64_t tick_ps, DevState *st, int ncu, hipStream_t s);
// Capacity-mode frame cache (hbf_cache.hip).  Caches of up to
// CACHE_LDS_MAX frames: the page held by each frame (-1 empty) and a
// prefetched-and-not-yet-hit flag per frame, loaded into LDS per call.
// Larger caches: the number of each page's latest insertion (PINS_NEVER if
// none) and, per frame, a prefetched flag and a hit-since-insertion flag.
// Both: the FIFO head, the counters (hits, faults, prefetch reads,
// prefetched used, evicted unused), the insertion count and the prefetched
// pages resident and unhit (device-memory caches, after each run).
struct CacheCtl {
  uint32_t head;
  uint32_t pad;
  int64_t count[5];
  int64_t ins;
  int64_t pend;
};
struct CacheCfg {
  int64_t *frame_page;
  uint32_t *frame_pf;
  int64_t *pins;
  uint8_t *fpf, *fhit;
  CacheCtl *ctl;
  uint32_t F, d;
};
constexpr int64_t PINS_NEVER = INT64_MIN / 4;
// Chunked solve of a device-memory cache (hbf_cache_chunk.hip).  Per page
// (R entries each, tagged with the chunk's epoch in the high 32 bits): the
// chunk's first access (tag ~epoch, kept by atomicMin), its last access,
// and, for a page inserted by the chunk, the time of the fault that
// inserted it (bits 0-23) and its rank among that fault's insertions (bits
// 24-29).  Per chunk: the per-access insertion/fault counts and their
// exclusive scan (S, Lmax + 1 entries), the sums per 1,024 accesses and
// the segment starts.
struct ChunkCtl {
  uint32_t nseg, valid;
  int64_t I0, npf0;  // insertions and prefetch outputs before the chunk
  int64_t lost_old;  // frames filled before the chunk, evicted within it holding a prefetched page never hit
};
struct ChunkCfg {
  uint64_t *at, *lt, *tt;
  uint64_t *S;
  uint64_t *bs;
  uint32_t *seg;
  ChunkCtl *ctl;
  uint32_t Lmax;
};
constexpr uint32_t CHUNK_MAX = 1u << 18;          // accesses per chunk
constexpr uint64_t CHUNK_MAX_R = uint64_t(1) << 26;  // range pages with per-page chunk state
constexpr uint32_t CHUNK_MIN = 16384;            // default accesses per chunk, at least

constexpr uint32_t CACHE_MAX_PREFETCH = 63;  // one fault's candidates fit one wave
// Caches of up to this many frames run with their whole state in LDS (a
// hash of the resident pages); larger ones keep each page's latest
// insertion number in device memory, which needs at least 64 frames (a
// round of 64 accesses without prefetch then never evicts a page it
// inserted, and one fault's insertion offsets, at most 63, stay below F).
constexpr uint32_t CACHE_LDS_MAX = 63;
// Default accesses per chunk for F frames (0: sequential only).  A chunk
// whose check fails costs its sequential run plus a few launches, so the
// default is long; F/16 above the minimum keeps a large cache's chunks from
// turning over its whole window.
inline uint32_t chunk_default(uint32_t F, uint64_t R) {
  if (F <= CACHE_LDS_MAX || R > CHUNK_MAX_R) return 0;
  uint32_t c = F / 16;
  return c < CHUNK_MIN ? CHUNK_MIN : (c > CHUNK_MAX ? CHUNK_MAX : c);
}
hipError_t launch_cache_clear(CacheCfg *dev_cfgs, int n_cfg, uint64_t R, uint32_t max_f, hipStream_t s);
// cfg_ids: the caches to run (device, n_cfg entries); every one of them has
// F <= CACHE_LDS_MAX when lds is set, else F > CACHE_LDS_MAX.  max_f: their
// largest frame count.
hipError_t launch_cache_run(const CacheCfg *dev_cfgs, const int *cfg_ids, int n_cfg, bool lds, uint32_t max_f,
                            uint64_t R, const uint64_t *pages, int64_t n, uint8_t *hit, uint64_t *pf_page,
                            int64_t *pf_src, int64_t pf_cap, int64_t *status, int64_t *n_pf_out, hipStream_t s);
// The sequential device-memory run alone (no page check, no pending count):
// caches whose chunk check passed (ccfgs[id].ctl->valid) are skipped; the
// prefetch outputs continue from *n_pf_out and name access i_base + i.
hipError_t launch_cache_seq(const CacheCfg *dev_cfgs, const ChunkCfg *dev_ccfgs, const int *cfg_ids, int n_cfg,
                            uint64_t R, const uint64_t *pages, int64_t n, int64_t i_base, uint8_t *hit,
                            uint64_t *pf_page, int64_t *pf_src, int64_t pf_cap, const int64_t *status,
                            int64_t *n_pf_out, hipStream_t s);
hipError_t cache_set_lds_limit();
// One chunk pages[c0 .. c0 + L) of the caches ids[0..n_cfg) (all with chunk
// state, L <= their Lmax): parallel solve, check, commit or undo, then the
// sequential run for the caches whose check failed.  epoch: nonzero, new
// for every chunk since the tags were cleared.
hipError_t launch_cache_chunk(const CacheCfg *dev_cfgs, const ChunkCfg *dev_ccfgs, const int *cfg_ids, int n_cfg,
                              uint32_t max_f, uint32_t max_d, uint64_t R, const uint64_t *pages, int64_t c0,
                              int64_t L, uint32_t epoch, uint8_t *hit, uint64_t *pf_page, int64_t *pf_src,
                              int64_t pf_cap, int64_t *status, int64_t *n_pf, hipStream_t s);
hipError_t launch_cache_check(const uint64_t *pages, int64_t n, uint64_t R, int64_t *status, hipStream_t s);
hipError_t launch_cache_pending(const CacheCfg *dev_cfgs, const int *cfg_ids, int n_cfg, uint32_t max_f,
                                const int64_t *status, hipStream_t s);
hipError_t launch_chunk_clear(const ChunkCfg *dev_ccfgs, const int *cfg_ids, int n_cfg, uint64_t R, hipStream_t s);
hipError_t launch_cache_report(const CacheCfg *dev_cfgs, int n_cfg, const int64_t *n_pf, const int64_t *status,
                               int64_t *out, int per_cfg, hipStream_t s);

extern const char *const kKernelNames[];
extern const int kNumTimedKernels;

}  // namespace hbf
