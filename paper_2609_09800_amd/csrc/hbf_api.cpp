// C ABI of the HBF hot path: argument validation, range snapshots,
// workspace management and kernel orchestration.  No torch types; the caller
// passes device pointers and a hipStream_t.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>
#include <tuple>
#include <vector>

#include "hbf.h"
#include "hbf_internal.h"

namespace hbf {
hipError_t set_lds_limits(uint32_t K);

static size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

Layout make_layout(const Geo &g, int64_t n) {
  Layout L{};
  L.n = n;
  if (g.vmem) {  // the vmem route: tile summaries and one service per request
    const size_t nt = (size_t)((n + VM_TILE - 1) / VM_TILE);
    size_t o = 0;
    L.off_ctl = o;   o = up256(o + sizeof(CallCtl));
    L.off_vsum = o;  o = up256(o + nt * 32);
    L.off_vin = o;   o = up256(o + nt * 32);
    L.off_vpair = o; o = up256(o + nt * 16);
    L.off_vfin = o;  o = up256(o + nt * 8);
    L.off_vcost = o; o = up256(o + (size_t)n * 4);
    L.off_vend = o;  o = up256(o + 64);
    L.off_vwsum = o; o = up256(o + nt * (VM_THREADS / 64) * 32);
    L.off_vwpair = o; o = up256(o + nt * (VM_THREADS / 64) * 16);
    L.total = o;
    return L;
  }
  int64_t te = (n + TARGET_TILES - 1) / TARGET_TILES;
  te = ((te + CHUNK - 1) / CHUNK) * CHUNK;
  if (te < CHUNK) te = CHUNK;
  L.tile_elems = te;
  L.nt = (uint32_t)((n + te - 1) / te);
  if (L.nt == 0) L.nt = 1;
  // cell width 2^s0 = Ts * 2^floor(log2 tR) <= Ts * tR keeps a cell at <= Ts
  // requests per die queue and at Ts time buckets
  int64_t Ts = 1;
  while (Ts * 2 <= MAX_BUCKETS && Ts * 2 * g.Dk <= MCAP) Ts *= 2;
  uint32_t lt = 0;
  while (Ts > 1 && (int64_t(1) << (lt + 1)) <= Ts) lt++;
  L.s0 = g.lg_tR + lt;
  const int64_t per = (int64_t)g.C * g.Dk * Ts;
  int64_t gm = 4 * ((n + per - 1) / per);
  if (gm < 64) gm = 64;
  L.gmax = (uint32_t)gm;
  const size_t K = g.K, nt = L.nt, C = g.C;
  size_t o = 0;
  L.off_ctl = o;      o = up256(o + sizeof(CallCtl));
  L.off_agg_cnt = o;  o = up256(o + nt * K * 4);
  L.off_agg_A = o;    o = up256(o + nt * K * 8);
  L.off_tin_L = o;    o = up256(o + nt * K * 8);
  L.off_tin_base = o; o = up256(o + nt * K * 4);
  L.off_totals = o;   o = up256(o + K * 4);
  L.off_seg = o;      o = up256(o + K * 4);
  L.off_dfnew = o;    o = up256(o + K * 8);
  L.off_cfnew = o;    o = up256(o + C * 8);
  L.off_dd = o;       o = up256(o + (size_t)n * 8);
  L.off_ix = o;       o = up256(o + (size_t)n * 4);
  L.off_kr = o;       o = up256(o + (size_t)n * 4);
  L.off_lb = o;       o = up256(o + C * ((size_t)L.gmax + 1) * g.Dk * 4);
  L.off_cagg = o;     o = up256(o + C * (size_t)L.gmax * 8);
  L.off_cgin = o;     o = up256(o + C * (size_t)L.gmax * 8);
  L.off_wst = o;      o = up256(o + 2 * C * (size_t)L.gmax * 8);
  L.off_nbl = o;      o = up256(o + C * (size_t)L.gmax * 4);
  L.off_iss = o;      o = up256(o + (g.reg_block ? (size_t)n * 8 : 0));
  L.total = o;
  return L;
}
}  // namespace hbf

using namespace hbf;

struct hbf_model {
  hbf_params p;
  Geo g;
  std::vector<uint64_t> rbase, rbytes, rpbase;  // registration order
  uint64_t total_pages = 0;
  int dev = -1;
  DevState *st = nullptr;
  void *ws = nullptr;
  size_t ws_cap = 0;
  bool ws_caller = false;
  bool lib_ws = false;
  bool prof = false;
  static constexpr int RING = 64;      // profiled calls kept
  hipEvent_t ev[RING][16] = {};
  int prof_calls = 0;                  // calls recorded since hbf_profile(.., 1)
  int ncu = 0;
  int64_t tick_ps = 0;
  // refresh: tPROG (-1 = not configured); per die queue, the completion
  // cells of the quanta uploaded last (the device consumes a prefix of each
  // list); whether quanta may still be pending on the device
  int64_t t_prog = -1;
  std::vector<std::vector<int64_t *>> ref_q;
  bool ref_maybe = false;
  int64_t **ref_slot = nullptr;
  size_t ref_slot_cap = 0;
  // closed-loop layers in one launch: library-owned scratch, the host copy
  // of each call's layer and tile lists and an event after its upload, and
  // whether the geometry can take that path on this GPU (-1: not asked yet)
  void *lay_ws = nullptr;
  size_t lay_cap = 0;
  std::vector<unsigned char> lay_up;
  hipEvent_t lay_ev = nullptr;
  int lay_ok = -1;
};

static bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }
static uint32_t lg2(uint64_t x) {
  uint32_t r = 0;
  while ((uint64_t(1) << r) < x) r++;
  return r;
}

static int ensure_device(hbf_model *m) {
  if (m->st) return HBF_OK;
  if (hipGetDevice(&m->dev) != hipSuccess) return HBF_EHIP;
  void *p = nullptr;
  if (hipMalloc(&p, sizeof(DevState)) != hipSuccess) return HBF_ENOMEM;
  m->st = (DevState *)p;
  std::vector<DevState> host(1);
  for (int k = 0; k < MAX_KEYS; k++) host[0].die_free[k] = NEG;
  for (int c = 0; c < MAX_CHANNELS; c++) host[0].chan_free[c] = NEG;
  host[0].sticky = 0;
  host[0].pad = 0;
  host[0].gemv_origin = 0;
  host[0].vfree = NEG;
  host[0].vlast = 0;
  host[0].vburst = 0;
  host[0].vhave = 0;
  host[0].vpad = 0;
  if (hipMemcpy(m->st, host.data(), sizeof(DevState), hipMemcpyHostToDevice) != hipSuccess) return HBF_EHIP;
  // (for the largest die-queue count: models of any size may follow)
  if (set_lds_limits(MAX_KEYS) != hipSuccess) return HBF_EHIP;
  if (hipDeviceGetAttribute(&m->ncu, hipDeviceAttributeMultiprocessorCount, m->dev) != hipSuccess)
    return HBF_EHIP;
  int rate_khz = 0;
  if (hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, m->dev) != hipSuccess ||
      rate_khz <= 0)
    return HBF_EHIP;
  m->tick_ps = 1000000000LL / rate_khz;
  return HBF_OK;
}

// (no heap allocation: the no-allocation entry point takes snapshots too)
static RangeTable snapshot(const hbf_model *m) {
  RangeTable rt;
  std::memset(&rt, 0, sizeof(rt));
  const int n = (int)m->rbase.size();
  int idx[MAX_RANGES];
  for (int i = 0; i < n; i++) idx[i] = i;
  std::sort(idx, idx + n, [&](int a, int b) { return m->rbase[a] < m->rbase[b]; });
  for (int i = 0; i < n; i++) {
    rt.base[i] = m->rbase[idx[i]];
    rt.bytes[i] = m->rbytes[idx[i]];
    rt.pbase[i] = m->rpbase[idx[i]];
    rt.rid[i] = (uint32_t)idx[i];
  }
  rt.n = n;
  return rt;
}

extern "C" {

int hbf_model_create(const hbf_params *params, hbf_model_t *out) {
  if (!params || !out) return HBF_EINVAL;
  const hbf_params &p = *params;
  if (p.channels < 1 || p.channels > 1024) return HBF_EINVAL;
  if (p.dies_per_channel < 1 || p.dies_per_channel > 256) return HBF_EINVAL;
  if (p.planes_per_die < 1 || p.planes_per_die > 64) return HBF_EINVAL;
  if (p.page_bytes == 0) return HBF_EINVAL;
  if (p.t_read_ns < 1 || p.t_read_ns > SERVICE_LIMIT) return HBF_EINVAL;
  if (p.channel_bytes_per_s == 0) return HBF_EINVAL;
  if (p.flags & ~(HBF_FLAG_PLANE_PARALLEL | HBF_FLAG_REGISTER_BLOCKING | HBF_FLAG_VMEM_CURVE)) return HBF_EINVAL;
  if ((p.flags & HBF_FLAG_VMEM_CURVE) && (p.flags & HBF_FLAG_REGISTER_BLOCKING)) return HBF_EINVAL;
  const uint64_t cdp = (uint64_t)p.channels * p.dies_per_channel * p.planes_per_die;
  if (cdp > 65536) return HBF_EINVAL;
  const bool pp = (p.flags & HBF_FLAG_PLANE_PARALLEL) != 0;
  const uint64_t Dk = (uint64_t)p.dies_per_channel * (pp ? p.planes_per_die : 1);
  const uint64_t K = (uint64_t)p.channels * Dk;
  if (Dk > MAX_RUNS || K > MAX_KEYS) return HBF_EINVAL;
  const unsigned __int128 num = (unsigned __int128)p.page_bytes * 1000000000u;
  const unsigned __int128 q = (num + p.channel_bytes_per_s - 1) / p.channel_bytes_per_s;
  if (q < 1 || q > (unsigned __int128)SERVICE_LIMIT) return HBF_EINVAL;
  hbf_model *m = new (std::nothrow) hbf_model();
  if (!m) return HBF_ENOMEM;
  m->p = p;
  Geo &g = m->g;
  g.C = p.channels;
  g.D = p.dies_per_channel;
  g.P = p.planes_per_die;
  g.Dk = (uint32_t)Dk;
  g.K = (uint32_t)K;
  g.page_bytes = p.page_bytes;
  g.plane_parallel = pp;
  g.reg_block = (p.flags & HBF_FLAG_REGISTER_BLOCKING) != 0;
  g.vmem = (p.flags & HBF_FLAG_VMEM_CURVE) != 0;
  {  // until configured: every page of a burst at the printed single-page cost
    const int64_t kp[6] = {1, 4, 16, 64, 256, 512};
    for (int k = 0; k < 6; k++) g.vknot[k] = 11133 * kp[k];
  }
  g.pow2 = is_pow2(p.page_bytes) && is_pow2(p.channels) && is_pow2(p.dies_per_channel) &&
           is_pow2(p.planes_per_die);
  g.lg_page = lg2(p.page_bytes);
  g.lg_C = lg2(p.channels);
  g.lg_D = lg2(p.dies_per_channel);
  g.lg_P = lg2(p.planes_per_die);
  g.tR = p.t_read_ns;
  g.lg_tR = 0;
  while ((int64_t(1) << (g.lg_tR + 1)) <= p.t_read_ns) g.lg_tR++;
  g.xfer = (int64_t)q;
  *out = m;
  return HBF_OK;
}

void hbf_model_destroy(hbf_model_t m) {
  if (!m) return;
  if (m->st) {
    hipDeviceSynchronize();
    hipFree(m->st);
  }
  if (m->ws && m->lib_ws) hipFree(m->ws);
  if (m->lay_ws) hipFree(m->lay_ws);
  if (m->lay_ev) hipEventDestroy(m->lay_ev);
  if (m->ref_slot) hipFree(m->ref_slot);
  for (auto &set : m->ev)
    for (auto &e : set)
      if (e) hipEventDestroy(e);
  delete m;
}

int hbf_xfer_ns(hbf_model_t m, int64_t *x) {
  if (!m || !x) return HBF_EINVAL;
  *x = m->g.xfer;
  return HBF_OK;
}

int hbf_n_die_queues(hbf_model_t m, uint32_t *n) {
  if (!m || !n) return HBF_EINVAL;
  *n = m->g.K;
  return HBF_OK;
}

int hbf_model_reset(hbf_model_t m, void *stream) {
  if (!m) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  for (auto &q : m->ref_q) q.clear();
  m->ref_maybe = false;
  return launch_reset(m->st, (hipStream_t)stream) == hipSuccess ? HBF_OK : HBF_EHIP;
}

int hbf_register_range(hbf_model_t m, uint64_t base, uint64_t bytes, int32_t *range_id) {
  if (!m || bytes == 0) return HBF_EINVAL;
  if ((int)m->rbase.size() >= MAX_RANGES) return HBF_EINVAL;
  if (base % m->p.page_bytes || bytes % m->p.page_bytes) return HBF_EALIGN;
  if (base + bytes < base) return HBF_EINVAL;
  for (size_t r = 0; r < m->rbase.size(); r++) {
    const uint64_t b = m->rbase[r], e = b + m->rbytes[r];
    if (base < e && b < base + bytes) return HBF_EOVERLAP;
  }
  if (range_id) *range_id = (int32_t)m->rbase.size();
  m->rbase.push_back(base);
  m->rbytes.push_back(bytes);
  m->rpbase.push_back(m->total_pages);
  m->total_pages += bytes / m->p.page_bytes;
  return HBF_OK;
}

int hbf_workspace_bytes(hbf_model_t m, int64_t n, size_t *bytes) {
  if (!m || !bytes || n < 0 || n > N_LIMIT) return HBF_EINVAL;
  *bytes = make_layout(m->g, n).total;
  return HBF_OK;
}

int hbf_set_workspace(hbf_model_t m, void *dev_ptr, size_t bytes) {
  if (!m) return HBF_EINVAL;
  if ((dev_ptr == nullptr) != (bytes == 0)) return HBF_EINVAL;
  if ((uintptr_t)dev_ptr % 256) return HBF_EINVAL;
  if (m->ws && m->lib_ws) {
    hipDeviceSynchronize();
    hipFree(m->ws);
  }
  m->ws = dev_ptr;
  m->ws_cap = bytes;
  m->ws_caller = dev_ptr != nullptr;
  m->lib_ws = false;
  return HBF_OK;
}

int hbf_classify_map(hbf_model_t m, const uint64_t *addr, int64_t n, uint64_t *map, void *stream) {
  if (!m || n < 0 || n > N_LIMIT || (n > 0 && (!addr || !map))) return HBF_EINVAL;
  if (m->g.C > 1024 || m->g.D > 256 || m->g.P > 64) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (n == 0) return HBF_OK;
  RangeTable rt = snapshot(m);
  return launch_classify(m->g, rt, m->st, addr, n, map, (hipStream_t)stream) == hipSuccess ? HBF_OK
                                                                                         : HBF_EHIP;
}

// Workspace for calls of up to n requests (grows library-owned scratch).
static int ensure_ws(hbf_model_t m, int64_t n) {
  const Layout L = make_layout(m->g, n);
  if (m->ws_caller) return m->ws_cap < L.total ? HBF_ENOWORKSPACE : HBF_OK;
  if (m->ws_cap >= L.total) return HBF_OK;
  if (m->ws) {
    hipDeviceSynchronize();
    hipFree(m->ws);
    m->ws = nullptr;
    m->ws_cap = 0;
  }
  void *p = nullptr;
  if (hipMalloc(&p, L.total) != hipSuccess) return HBF_ENOMEM;
  m->ws = p;
  m->ws_cap = L.total;
  m->lib_ws = true;
  return HBF_OK;
}

// Enqueue one timing call (workspace already sized for n > 0).
static int time_call(hbf_model_t m, const RangeTable &rt, const uint64_t *addr, const int64_t *issue,
                     int64_t n, int64_t *complete, void *stream) {
  const Layout L = make_layout(m->g, n);
  hipEvent_t *ev = nullptr;
  if (m->prof && !m->g.vmem) {  // (per-kernel timing covers the media model's kernels)
    hipEvent_t *set = m->ev[m->prof_calls % hbf_model::RING];
    for (int k = 0; k <= kNumTimedKernels; k++)
      if (!set[k] && hipEventCreate(&set[k]) != hipSuccess) return HBF_EHIP;
    ev = set;
  }
  hipError_t e = launch_time_requests(m->g, rt, L, (char *)m->ws, m->st, addr, issue, complete,
                                      (hipStream_t)stream, ev, kNumTimedKernels + 1, m->ref_maybe);
  if (e != hipSuccess) return HBF_EHIP;
  if (ev) m->prof_calls++;
  return HBF_OK;
}

int hbf_time_requests(hbf_model_t m, const uint64_t *addr, const int64_t *issue, int64_t n,
                      int64_t *complete, void *stream) {
  if (!m || n < 0 || n > N_LIMIT || (n > 0 && (!addr || !issue || !complete))) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (n == 0) return HBF_OK;
  if ((rc = ensure_ws(m, n))) return rc;
  return time_call(m, snapshot(m), addr, issue, n, complete, stream);
}

int hbf_time_requests_noalloc(hbf_model_t m, const uint64_t *addr, const int64_t *issue, int64_t n,
                              int64_t *complete, void *stream) {
  if (!m || n < 0 || n > N_LIMIT || (n > 0 && (!addr || !issue || !complete))) return HBF_EINVAL;
  int dev = -1;
  if (!m->st || hipGetDevice(&dev) != hipSuccess || dev != m->dev) return HBF_EINVAL;
  if (n == 0) return HBF_OK;
  const Layout L = make_layout(m->g, n);
  if (L.total > HBF_NOALLOC_SCRATCH_BYTES) return HBF_ENOWORKSPACE;
  char *ws = nullptr;
  if (noalloc_scratch(dev, &ws) != hipSuccess) return HBF_EHIP;
  return launch_time_requests(m->g, snapshot(m), L, ws, m->st, addr, issue, complete, (hipStream_t)stream,
                              nullptr, 0, m->ref_maybe) == hipSuccess
             ? HBF_OK
             : HBF_EHIP;
}

int hbf_time_layers(hbf_model_t m, const uint64_t *addr, int64_t n, const int64_t *ls, int L,
                    int64_t t_start, int64_t compute_ns, int64_t *issue, int64_t *complete, int64_t *done,
                    void *stream) {
  if (!m || n < 0 || n > N_LIMIT || L < 0 || !ls) return HBF_EINVAL;
  if (t_start < 0 || t_start >= ISSUE_LIMIT || compute_ns < 0 || compute_ns >= ISSUE_LIMIT) return HBF_EINVAL;
  if (ls[0] != 0 || ls[L] != n) return HBF_EINVAL;
  int64_t most = 0;
  for (int l = 0; l < L; l++) {
    if (ls[l + 1] < ls[l]) return HBF_EINVAL;
    most = std::max(most, ls[l + 1] - ls[l]);
  }
  if (L > 0 && !done) return HBF_EINVAL;
  if (n > 0 && (!addr || !issue || !complete)) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (L == 0) return HBF_OK;
  const RangeTable rt = snapshot(m);
  const hipStream_t s = (hipStream_t)stream;
  // One launch for all layers when nothing but the plain two-stage model is
  // involved (no refresh quanta pending, no register blocking, not the vmem
  // route), the library owns the scratch, and every channel's workgroup can
  // be resident at once; otherwise one timing call per layer.
  if (m->lay_ok < 0) m->lay_ok = layers_fast_ok(m->g, m->ncu) ? 1 : 0;
  if (!m->ref_maybe && !m->g.reg_block && !m->g.vmem && !m->ws_caller && most <= LAYERS_MAX_LAYER &&
      L <= LAYERS_MAX_COUNT && m->lay_ok) {
    if (!m->lay_ev) {
      if (hipEventCreateWithFlags(&m->lay_ev, hipEventDisableTiming) != hipSuccess) return HBF_EHIP;
      if (hipEventRecord(m->lay_ev, s) != hipSuccess) return HBF_EHIP;
    }
    const size_t need = layers_ws_bytes(m->g, n, L);
    if (m->lay_cap < need) {
      if (m->lay_ws) {
        hipDeviceSynchronize();
        hipFree(m->lay_ws);
        m->lay_ws = nullptr;
        m->lay_cap = 0;
      }
      void *p = nullptr;
      if (hipMalloc(&p, need) != hipSuccess) return HBF_ENOMEM;
      m->lay_ws = p;
      m->lay_cap = need;
    }
    if (launch_layers(m->g, rt, (char *)m->lay_ws, m->st, addr, n, ls, L, t_start, compute_ns, issue, complete,
                      done, m->lay_up, m->lay_ev, s) != hipSuccess)
      return HBF_EHIP;
    return HBF_OK;
  }
  if (most > 0 && (rc = ensure_ws(m, most))) return rc;
  for (int l = 0; l < L; l++) {
    const int64_t a = ls[l], cnt = ls[l + 1] - ls[l];
    const int64_t *prev = l > 0 ? done + (l - 1) : nullptr;
    if (launch_layer_issue(issue + a, cnt, prev, t_start, compute_ns, s) != hipSuccess) return HBF_EHIP;
    if (cnt > 0 && (rc = time_call(m, rt, addr + a, issue + a, cnt, complete + a, stream))) return rc;
    // the control block of the call just enqueued; read only when cnt > 0
    const CallCtl *ctl = cnt > 0 ? reinterpret_cast<const CallCtl *>((char *)m->ws + make_layout(m->g, cnt).off_ctl)
                                 : nullptr;
    if (launch_layer_done(ctl, cnt, prev, t_start, compute_ns, done + l, s) != hipSuccess) return HBF_EHIP;
  }
  return HBF_OK;
}

// ---- refresh (Section D4)

// Die queue of device page p (channel-first striping).
static uint32_t key_of_page(const Geo &g, uint64_t p) {
  const uint32_t ch = (uint32_t)(p % g.C), die = (uint32_t)((p / g.C) % g.D);
  const uint32_t plane = (uint32_t)((p / ((uint64_t)g.C * g.D)) % g.P);
  const uint32_t k = ch * g.D + die;
  return g.plane_parallel ? k * g.P + plane : k;
}

int hbf_refresh_plan(const hbf_params *params, const hbf_refresh_block *blocks, int64_t n_blocks,
                     uint32_t ppb, uint64_t *out, int64_t cap) {
  if (!params || n_blocks < 0 || (n_blocks > 0 && (!blocks || !out)) || ppb < 1) return HBF_EINVAL;
  const uint64_t C = params->channels, D = params->dies_per_channel, P = params->planes_per_die;
  if (C < 1 || D < 1 || P < 1) return HBF_EINVAL;
  if ((unsigned __int128)n_blocks * ppb > (unsigned __int128)cap) return HBF_EINVAL;
  for (int64_t b = 0; b < n_blocks; b++)
    if (blocks[b].channel >= C || blocks[b].die >= D || blocks[b].plane >= P) return HBF_EINVAL;
  std::vector<int64_t> idx(n_blocks);
  for (int64_t b = 0; b < n_blocks; b++) idx[b] = b;
  // a physical block is eligible at most once per epoch: the order places
  // each eligible block once, so a block listed twice in an epoch is refused
  {
    auto phys = [&](int64_t x) {
      const hbf_refresh_block &a = blocks[x];
      return std::make_tuple(a.epoch, a.channel, a.die, a.plane, a.block);
    };
    std::sort(idx.begin(), idx.end(), [&](int64_t x, int64_t y) { return phys(x) < phys(y); });
    for (int64_t i = 1; i < n_blocks; i++)
      if (phys(idx[i - 1]) == phys(idx[i])) return HBF_EINVAL;
  }
  // per epoch: each die's pages in (zone, block, plane, page) order
  std::sort(idx.begin(), idx.end(), [&](int64_t x, int64_t y) {
    const hbf_refresh_block &a = blocks[x], &c = blocks[y];
    if (a.epoch != c.epoch) return a.epoch < c.epoch;
    if (a.zone != c.zone) return a.zone < c.zone;
    if (a.block != c.block) return a.block < c.block;
    if (a.plane != c.plane) return a.plane < c.plane;
    return x < y;
  });
  int64_t w = 0;
  for (int64_t e0 = 0; e0 < n_blocks;) {
    int64_t e1 = e0;
    while (e1 < n_blocks && blocks[idx[e1]].epoch == blocks[idx[e0]].epoch) e1++;
    // die (c, d) -> its blocks of this epoch in order; cursor in pages
    std::vector<std::vector<int64_t>> die_blocks(C * D);
    for (int64_t i = e0; i < e1; i++) {
      const hbf_refresh_block &b = blocks[idx[i]];
      die_blocks[(uint64_t)b.channel * D + b.die].push_back(idx[i]);
    }
    std::vector<uint64_t> cur(C * D, 0), left(C * D, 0);
    std::vector<uint64_t> chan_left(C, 0);
    for (uint64_t cd = 0; cd < C * D; cd++) {
      left[cd] = (uint64_t)die_blocks[cd].size() * ppb;
      chan_left[cd / D] += left[cd];
    }
    std::vector<int64_t> last(C, -1);
    uint64_t total = (uint64_t)(e1 - e0) * ppb;
    while (total) {
      for (uint64_t c = 0; c < C; c++) {
        if (!chan_left[c]) continue;
        // next die after the last served one, cyclically, with pages left
        uint64_t d = (uint64_t)(last[c] + 1) % D;
        while (!left[c * D + d]) d = (d + 1) % D;
        const uint64_t cd = c * D + d;
        const hbf_refresh_block &b = blocks[die_blocks[cd][cur[cd] / ppb]];
        const uint64_t pg = (uint64_t)b.block * ppb + cur[cd] % ppb;
        out[w++] = ((pg * P + b.plane) * D + d) * C + c;
        cur[cd]++;
        left[cd]--;
        chan_left[c]--;
        total--;
        last[c] = (int64_t)d;
      }
    }
    e0 = e1;
  }
  return HBF_OK;
}

int hbf_vmem_configure(hbf_model_t m, const int64_t *knot) {
  if (!m || !knot || !m->g.vmem) return HBF_EINVAL;
  const int64_t kp[6] = {1, 4, 16, 64, 256, 512};
  if (knot[0] < 1 || knot[0] > SERVICE_LIMIT) return HBF_EINVAL;
  for (int k = 1; k < 6; k++) {
    if (knot[k] < knot[k - 1]) return HBF_EINVAL;
    if (knot[k] - knot[k - 1] > SERVICE_LIMIT * (kp[k] - kp[k - 1])) return HBF_EINVAL;
  }
  for (int k = 0; k < 6; k++) m->g.vknot[k] = knot[k];
  return HBF_OK;
}

int hbf_refresh_configure(hbf_model_t m, int64_t t_prog_ns) {
  if (!m || m->g.vmem || t_prog_ns < 0 || 2 * m->g.tR + t_prog_ns > SERVICE_LIMIT) return HBF_EINVAL;
  m->t_prog = t_prog_ns;
  m->g.tQ = m->g.tR + t_prog_ns;
  return HBF_OK;
}

int hbf_refresh_submit(hbf_model_t m, const uint64_t *pages, int64_t nq, int64_t *done, void *stream) {
  if (!m || m->t_prog < 0 || nq < 0 || nq > N_LIMIT || (nq > 0 && (!pages || !done))) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  const uint32_t K = m->g.K;
  const hipStream_t s = (hipStream_t)stream;
  if (m->ref_q.size() != K) m->ref_q.assign(K, {});
  // what the device consumed of the lists uploaded last
  std::vector<uint32_t> head(K), pend(K);
  if (hipStreamSynchronize(s) != hipSuccess ||
      hipMemcpy(head.data(), m->st->ref_head, K * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(pend.data(), m->st->ref_pend, K * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return HBF_EHIP;
  uint64_t total = nq;
  for (uint32_t k = 0; k < K; k++) {
    std::vector<int64_t *> &q = m->ref_q[k];
    if ((uint64_t)head[k] + pend[k] > q.size()) return HBF_EHIP;  // device state out of step
    q.erase(q.begin(), q.begin() + head[k]);
    q.resize(pend[k]);
    total += q.size();
  }
  if (total > (uint64_t)UINT32_MAX) return HBF_EINVAL;
  for (int64_t j = 0; j < nq; j++) m->ref_q[key_of_page(m->g, pages[j])].push_back(done + j);
  // flatten: die queue k's pending cells at [off[k], off[k] + pend[k])
  std::vector<int64_t *> flat;
  flat.reserve(total);
  std::vector<uint32_t> off(K);
  for (uint32_t k = 0; k < K; k++) {
    off[k] = (uint32_t)flat.size();
    pend[k] = (uint32_t)m->ref_q[k].size();
    head[k] = 0;
    flat.insert(flat.end(), m->ref_q[k].begin(), m->ref_q[k].end());
  }
  if (flat.size() > m->ref_slot_cap) {
    if (m->ref_slot) hipFree(m->ref_slot);
    m->ref_slot = nullptr;
    m->ref_slot_cap = 0;
    void *p = nullptr;
    if (hipMalloc(&p, flat.size() * sizeof(int64_t *)) != hipSuccess) return HBF_ENOMEM;
    m->ref_slot = (int64_t **)p;
    m->ref_slot_cap = flat.size();
  }
  if ((!flat.empty() &&
       hipMemcpy(m->ref_slot, flat.data(), flat.size() * sizeof(int64_t *), hipMemcpyHostToDevice) != hipSuccess) ||
      hipMemcpy(&m->st->ref_slot, &m->ref_slot, sizeof(int64_t **), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(m->st->ref_off, off.data(), K * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(m->st->ref_head, head.data(), K * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(m->st->ref_pend, pend.data(), K * 4, hipMemcpyHostToDevice) != hipSuccess)
    return HBF_EHIP;
  if (launch_fill(done, nq, REFRESH_PENDING, s) != hipSuccess) return HBF_EHIP;
  m->ref_maybe = !flat.empty();
  return HBF_OK;
}

int hbf_refresh_drain(hbf_model_t m, int64_t t_from, int64_t t_to, void *stream) {
  if (!m || t_from < 0 || t_to < t_from || t_to >= ISSUE_LIMIT) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (!m->ref_maybe) return HBF_OK;
  return launch_refresh_drain(m->g, m->st, t_from, t_to, (hipStream_t)stream) == hipSuccess ? HBF_OK : HBF_EHIP;
}

int hbf_refresh_pending(hbf_model_t m, uint32_t *host_pending, void *stream) {
  if (!m || !host_pending) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess ||
      hipMemcpy(host_pending, m->st->ref_pend, m->g.K * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return HBF_EHIP;
  bool any = false;
  for (uint32_t k = 0; k < m->g.K; k++) any |= host_pending[k] != 0;
  m->ref_maybe = any;
  return HBF_OK;
}

// ---- capacity-mode frame cache (Sections D5, D6)

}  // extern "C"

struct hbf_cache {
  uint32_t F = 0, d = 0;
  uint64_t R = 0;
  void *mem = nullptr;         // frames | flags | slots | ctl | chunk state | cfg | status, n_pf
  CacheCfg *dcfg = nullptr;
  ChunkCfg *dccfg = nullptr;   // null when the cache has no chunk state
  int64_t *status = nullptr;   // [0] status, [1] prefetch reads of the call
  int *dids = nullptr;
  uint32_t lmax = 0;           // chunk state allocated for chunks of up to lmax accesses
  uint32_t chunk = 0;          // accesses per chunk; 0 = the sequential run alone
  uint32_t epoch = 0;          // last chunk tag used
};

static bool cache_params_ok(uint32_t F, uint32_t d, uint64_t R) {
  return F >= 1 && F < (1u << 31) && d < F && d <= CACHE_MAX_PREFETCH && R >= 1 && R <= (uint64_t)N_LIMIT;
}

struct CacheAlloc {
  void *mem = nullptr;
  CacheCfg *dcfg = nullptr;
  ChunkCfg *dccfg = nullptr;
  int64_t *status = nullptr;
  int *dids = nullptr;   // LDS caches, then sequential device-memory caches, then chunked ones
  int n_lds = 0, n_seq = 0, n_chunk = 0;
};

// Device state of n caches in one allocation.  lmax[b] > 0: cache b (a
// device-memory cache) also gets chunk state for chunks of up to lmax[b]
// accesses.
static int cache_alloc(const uint32_t *F, const uint32_t *d, const uint32_t *lmax, int n, uint64_t R,
                       CacheAlloc *out) {
  size_t o = 0;
  std::vector<size_t> off(n), coff(n);
  for (int b = 0; b < n; b++) {
    off[b] = o;
    if (F[b] <= CACHE_LDS_MAX) {  // frame pages and flags
      o = up256(o + (size_t)F[b] * 8);
      o = up256(o + (size_t)F[b] * 4);
    } else {  // latest insertion per page, two flags per frame
      o = up256(o + (size_t)R * 8);
      o = up256(o + (size_t)F[b]);
      o = up256(o + (size_t)F[b]);
    }
    o = up256(o + sizeof(CacheCtl));
    coff[b] = o;
    if (lmax[b]) {
      const size_t L = lmax[b];
      o = up256(o + R * 8 * 3);           // at, lt, tt
      o = up256(o + (L + 1) * 8);         // S
      o = up256(o + (L / 1024 + 1) * 8);  // bs
      o = up256(o + L * 4);               // seg
      o = up256(o + sizeof(ChunkCtl));
    }
  }
  const size_t oids = o;
  o = up256(o + sizeof(int) * n);
  const size_t ocfg = o;
  o = up256(o + sizeof(CacheCfg) * n);
  const size_t occfg = o;
  o = up256(o + sizeof(ChunkCfg) * n);
  const size_t ost = o;
  o = up256(o + 16);
  void *p = nullptr;
  if (hipMalloc(&p, o) != hipSuccess) return HBF_ENOMEM;
  char *base = (char *)p;
  std::vector<CacheCfg> cfg(n);
  std::vector<ChunkCfg> ccfg(n);
  for (int b = 0; b < n; b++) {
    size_t q = off[b];
    cfg[b] = CacheCfg{};
    if (F[b] <= CACHE_LDS_MAX) {
      cfg[b].frame_page = (int64_t *)(base + q);
      q = up256(q + (size_t)F[b] * 8);
      cfg[b].frame_pf = (uint32_t *)(base + q);
      q = up256(q + (size_t)F[b] * 4);
    } else {
      cfg[b].pins = (int64_t *)(base + q);
      q = up256(q + (size_t)R * 8);
      cfg[b].fpf = (uint8_t *)(base + q);
      q = up256(q + (size_t)F[b]);
      cfg[b].fhit = (uint8_t *)(base + q);
      q = up256(q + (size_t)F[b]);
    }
    cfg[b].ctl = (CacheCtl *)(base + q);
    cfg[b].F = F[b];
    cfg[b].d = d[b];
    ccfg[b] = ChunkCfg{};
    if (lmax[b]) {
      const size_t L = lmax[b];
      q = coff[b];
      ccfg[b].at = (uint64_t *)(base + q);
      ccfg[b].lt = ccfg[b].at + R;
      ccfg[b].tt = ccfg[b].lt + R;
      q = up256(q + R * 8 * 3);
      ccfg[b].S = (uint64_t *)(base + q);
      q = up256(q + (L + 1) * 8);
      ccfg[b].bs = (uint64_t *)(base + q);
      q = up256(q + (L / 1024 + 1) * 8);
      ccfg[b].seg = (uint32_t *)(base + q);
      q = up256(q + L * 4);
      ccfg[b].ctl = (ChunkCtl *)(base + q);
      ccfg[b].Lmax = lmax[b];
    }
  }
  std::vector<int> ids;
  for (int b = 0; b < n; b++)
    if (F[b] <= CACHE_LDS_MAX) ids.push_back(b);
  out->n_lds = (int)ids.size();
  for (int b = 0; b < n; b++)
    if (F[b] > CACHE_LDS_MAX && !lmax[b]) ids.push_back(b);
  out->n_seq = (int)ids.size() - out->n_lds;
  for (int b = 0; b < n; b++)
    if (F[b] > CACHE_LDS_MAX && lmax[b]) ids.push_back(b);
  out->n_chunk = n - out->n_lds - out->n_seq;
  if (hipMemcpy(base + ocfg, cfg.data(), sizeof(CacheCfg) * n, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(base + occfg, ccfg.data(), sizeof(ChunkCfg) * n, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(base + oids, ids.data(), sizeof(int) * n, hipMemcpyHostToDevice) != hipSuccess ||
      cache_set_lds_limit() != hipSuccess) {
    hipFree(p);
    return HBF_EHIP;
  }
  out->mem = p;
  out->dcfg = (CacheCfg *)(base + ocfg);
  out->dccfg = (ChunkCfg *)(base + occfg);
  out->status = (int64_t *)(base + ost);
  out->dids = (int *)(base + oids);
  return HBF_OK;
}

// Serve pages[0..n) on the chunked caches ids[0..n_chunk): chunk after chunk,
// each solved in parallel and checked, the sequential run for those that
// fail; then the prefetched pages still pending.  *epoch: the last tag used.
static bool run_chunks(const CacheCfg *dcfg, const ChunkCfg *dccfg, const int *ids, int n_chunk, uint32_t max_f,
                       uint32_t max_d, uint64_t R, const uint64_t *pages, int64_t n, uint32_t chunk,
                       uint32_t *epoch, uint8_t *hit, uint64_t *pf_page, int64_t *pf_src, int64_t pf_cap,
                       int64_t *status, int64_t *n_pf, hipStream_t s) {
  for (int64_t c0 = 0; c0 < n; c0 += chunk) {
    if (*epoch >= 0xFFFFFF00u) {  // tags about to repeat: clear them
      if (launch_chunk_clear(dccfg, ids, n_chunk, R, s) != hipSuccess) return false;
      *epoch = 0;
    }
    ++*epoch;
    const int64_t L = n - c0 < (int64_t)chunk ? n - c0 : (int64_t)chunk;
    if (launch_cache_chunk(dcfg, dccfg, ids, n_chunk, max_f, max_d, R, pages, c0, L, *epoch, hit, pf_page, pf_src,
                           pf_cap, status, n_pf, s) != hipSuccess)
      return false;
  }
  return launch_cache_pending(dcfg, ids, n_chunk, max_f, status, s) == hipSuccess;
}

extern "C" {

int hbf_cache_create(uint32_t frames, uint32_t prefetch_pages, uint64_t range_pages, hbf_cache_t *out) {
  if (!out || !cache_params_ok(frames, prefetch_pages, range_pages)) return HBF_EINVAL;
  hbf_cache *c = new (std::nothrow) hbf_cache();
  if (!c) return HBF_ENOMEM;
  c->F = frames;
  c->d = prefetch_pages;
  c->R = range_pages;
  c->lmax = frames > CACHE_LDS_MAX && range_pages <= CHUNK_MAX_R ? CHUNK_MAX : 0;
  c->chunk = chunk_default(frames, range_pages);
  CacheAlloc al;
  int rc = cache_alloc(&c->F, &c->d, &c->lmax, 1, c->R, &al);
  if (rc) {
    delete c;
    return rc;
  }
  c->mem = al.mem;
  c->dcfg = al.dcfg;
  c->dccfg = c->lmax ? al.dccfg : nullptr;
  c->status = al.status;
  c->dids = al.dids;
  bool ok = launch_cache_clear(c->dcfg, 1, c->R, c->F, nullptr) == hipSuccess;
  if (ok && c->dccfg) ok = launch_chunk_clear(c->dccfg, c->dids, 1, c->R, nullptr) == hipSuccess;
  if (!ok || hipDeviceSynchronize() != hipSuccess) {
    hipFree(c->mem);
    delete c;
    return HBF_EHIP;
  }
  *out = c;
  return HBF_OK;
}

void hbf_cache_destroy(hbf_cache_t c) {
  if (!c) return;
  hipDeviceSynchronize();
  hipFree(c->mem);
  delete c;
}

int hbf_cache_reset(hbf_cache_t c, void *stream) {
  if (!c) return HBF_EINVAL;
  return launch_cache_clear(c->dcfg, 1, c->R, c->F, (hipStream_t)stream) == hipSuccess ? HBF_OK : HBF_EHIP;
}

int hbf_cache_set_chunk(hbf_cache_t c, uint32_t accesses) {
  if (!c || (accesses && (!c->dccfg || accesses > c->lmax))) return HBF_EINVAL;
  c->chunk = accesses;
  return HBF_OK;
}

int hbf_cache_get_chunk(hbf_cache_t c, uint32_t *accesses) {
  if (!c || !accesses) return HBF_EINVAL;
  *accesses = c->chunk;
  return HBF_OK;
}

int hbf_cache_access(hbf_cache_t c, const uint64_t *pages, int64_t n, uint8_t *hit, uint64_t *pf_page,
                     int64_t *pf_src, int64_t pf_cap, int64_t *counts, void *stream) {
  if (!c || !counts || n < 0 || n > N_LIMIT || (n > 0 && (!pages || !hit))) return HBF_EINVAL;
  if ((pf_page == nullptr) != (pf_src == nullptr) || pf_cap < 0) return HBF_EINVAL;
  const hipStream_t s = (hipStream_t)stream;
  if (launch_fill(c->status, 2, 0, s) != hipSuccess) return HBF_EHIP;
  if (n > 0 && c->chunk) {
    if (launch_cache_check(pages, n, c->R, c->status, s) != hipSuccess ||
        !run_chunks(c->dcfg, c->dccfg, c->dids, 1, c->F, c->d, c->R, pages, n, c->chunk, &c->epoch, hit, pf_page,
                    pf_src, pf_page ? pf_cap : 0, c->status, c->status + 1, s))
      return HBF_EHIP;
  } else if (n > 0 && launch_cache_run(c->dcfg, c->dids, 1, c->F <= CACHE_LDS_MAX, c->F, c->R, pages, n, hit,
                                       pf_page, pf_src, pf_page ? pf_cap : 0, c->status, c->status + 1,
                                       s) != hipSuccess) {
    return HBF_EHIP;
  }
  return launch_cache_report(c->dcfg, 1, c->status + 1, c->status, counts, 8, s) == hipSuccess ? HBF_OK
                                                                                              : HBF_EHIP;
}

int hbf_cache_sweep(const uint32_t *frames, const uint32_t *prefetch, int n_cfg, uint64_t range_pages,
                    const uint64_t *pages, int64_t n, int64_t *counts, void *stream) {
  if (!frames || !prefetch || n_cfg < 1 || n_cfg > 65535 || !counts || n < 0 || n > N_LIMIT || (n > 0 && !pages))
    return HBF_EINVAL;
  uint32_t max_f = 0, chunk = 0;
  std::vector<uint32_t> lmax(n_cfg, 0);
  for (int b = 0; b < n_cfg; b++) {
    if (!cache_params_ok(frames[b], prefetch[b], range_pages)) return HBF_EINVAL;
    max_f = std::max(max_f, frames[b]);
    const uint32_t cd = chunk_default(frames[b], range_pages);
    if (cd) chunk = chunk ? std::min(chunk, cd) : cd;
  }
  // the chunked caches share one chunk length: the smallest of their defaults
  for (int b = 0; b < n_cfg; b++)
    if (chunk_default(frames[b], range_pages)) lmax[b] = chunk;
  CacheAlloc al;
  int rc = cache_alloc(frames, prefetch, lmax.data(), n_cfg, range_pages, &al);
  if (rc) return rc;
  const hipStream_t s = (hipStream_t)stream;
  uint32_t max_lds = 0, max_seq = 0, max_chunk = 0, max_dchunk = 0;
  for (int b = 0; b < n_cfg; b++) {
    if (frames[b] <= CACHE_LDS_MAX) max_lds = std::max(max_lds, frames[b]);
    else if (!lmax[b]) max_seq = std::max(max_seq, frames[b]);
    else {
      max_chunk = std::max(max_chunk, frames[b]);
      max_dchunk = std::max(max_dchunk, prefetch[b]);
    }
  }
  const int *ids_seq = al.dids + al.n_lds, *ids_chunk = al.dids + al.n_lds + al.n_seq;
  bool ok = launch_fill(al.status, 2, 0, s) == hipSuccess &&
            launch_cache_clear(al.dcfg, n_cfg, range_pages, max_f, s) == hipSuccess;
  if (ok && al.n_chunk) ok = launch_chunk_clear(al.dccfg, ids_chunk, al.n_chunk, range_pages, s) == hipSuccess;
  // the LDS-resident caches, the sequential device-memory ones, then the
  // chunked ones (all queued on the stream)
  if (ok && n > 0 && al.n_lds > 0)
    ok = launch_cache_run(al.dcfg, al.dids, al.n_lds, true, max_lds, range_pages, pages, n, nullptr, nullptr,
                          nullptr, 0, al.status, nullptr, s) == hipSuccess;
  if (ok && n > 0 && al.n_seq > 0)
    ok = launch_cache_run(al.dcfg, ids_seq, al.n_seq, false, max_seq, range_pages, pages, n, nullptr, nullptr,
                          nullptr, 0, al.status, nullptr, s) == hipSuccess;
  if (ok && n > 0 && al.n_chunk > 0) {
    uint32_t epoch = 0;
    ok = (al.n_lds + al.n_seq > 0 || launch_cache_check(pages, n, range_pages, al.status, s) == hipSuccess) &&
         run_chunks(al.dcfg, al.dccfg, ids_chunk, al.n_chunk, max_chunk, max_dchunk, range_pages, pages, n, chunk,
                    &epoch, nullptr, nullptr, nullptr, 0, al.status, nullptr, s);
  }
  ok = ok && launch_cache_report(al.dcfg, n_cfg, nullptr, al.status, counts, 5, s) == hipSuccess;
  // the temporary state is freed once the sweep has run
  ok = hipStreamSynchronize(s) == hipSuccess && ok;
  int64_t st = 0;
  ok = ok && hipMemcpy(&st, al.status, 8, hipMemcpyDeviceToHost) == hipSuccess;
  hipFree(al.mem);
  if (!ok) return HBF_EHIP;
  return st ? (int)st : HBF_OK;
}

int hbf_gemv_instrumented(hbf_model_t m, const uint16_t *W, int E, int K, int N, const uint16_t *X,
                          int B, float *Y, const int64_t *pi, const int64_t *pc, int64_t *meas,
                          void *stream) {
  if (!m || !W || !X || !Y || E < 1 || K < 1 || N < 1 || B < 1 || B > 64) return HBF_EINVAL;
  if ((pi == nullptr) != (pc == nullptr) || (meas && !pi)) return HBF_EINVAL;
  const uint64_t pb = m->p.page_bytes;
  if (K % 512 || K > 4096 || pb % ((uint64_t)K * 2)) return HBF_EINVAL;
  const uint64_t rows_per_page = pb / ((uint64_t)K * 2);
  if (rows_per_page > 16 || (uint64_t)N % rows_per_page) return HBF_EINVAL;
  if (((uintptr_t)W) % pb || ((uintptr_t)X) % 16 || ((uintptr_t)Y) % 4) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  return launch_gemv(W, E, K, N, (int)pb, X, B, Y, pi, pc, meas, m->tick_ps, m->st, m->ncu,
                     (hipStream_t)stream) == hipSuccess
             ? HBF_OK
             : HBF_EHIP;
}

int hbf_wall_clock_tick_ps(hbf_model_t m, int64_t *tick_ps) {
  if (!m || !tick_ps) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  *tick_ps = m->tick_ps;
  return HBF_OK;
}

int hbf_get_status(hbf_model_t m, void *stream) {
  if (!m) return HBF_EINVAL;
  if (!m->st) return HBF_OK;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return HBF_EHIP;
  uint32_t s = 0;
  if (hipMemcpy(&s, &m->st->sticky, 4, hipMemcpyDeviceToHost) != hipSuccess) return HBF_EHIP;
  const uint32_t z = 0;
  if (hipMemcpy(&m->st->sticky, &z, 4, hipMemcpyHostToDevice) != hipSuccess) return HBF_EHIP;
  if (s & (ERR_RANGE_TIME | ERR_OVERFLOW)) return HBF_ERANGE_TIME;
  if (s & ERR_UNSORTED) return HBF_EUNSORTED;
  if (s & ERR_MAP) return HBF_EINVAL;
  if (s & ERR_INTERNAL) return HBF_EINTERNAL;
  return HBF_OK;
}

int hbf_get_state(hbf_model_t m, int64_t *die_free, int64_t *chan_free, void *stream) {
  if (!m) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return HBF_EHIP;
  std::vector<DevState> h(1);
  if (hipMemcpy(h.data(), m->st, sizeof(DevState), hipMemcpyDeviceToHost) != hipSuccess) return HBF_EHIP;
  if (die_free)
    for (uint32_t k = 0; k < m->g.K; k++)
      die_free[k] = h[0].die_free[k] <= NEG ? INT64_MIN : h[0].die_free[k];
  if (chan_free)
    for (uint32_t c = 0; c < m->g.C; c++)
      chan_free[c] = h[0].chan_free[c] <= NEG ? INT64_MIN : h[0].chan_free[c];
  return HBF_OK;
}

int hbf_set_state(hbf_model_t m, const int64_t *die_free, const int64_t *chan_free, void *stream) {
  if (!m || !die_free || !chan_free) return HBF_EINVAL;
  for (uint32_t k = 0; k < m->g.K; k++)
    if (die_free[k] != INT64_MIN && (die_free[k] < 0 || die_free[k] >= TIME_LIMIT)) return HBF_EINVAL;
  for (uint32_t c = 0; c < m->g.C; c++)
    if (chan_free[c] != INT64_MIN && (chan_free[c] < 0 || chan_free[c] >= TIME_LIMIT)) return HBF_EINVAL;
  int rc = ensure_device(m);
  if (rc) return rc;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return HBF_EHIP;
  std::vector<DevState> h(1);
  if (hipMemcpy(h.data(), m->st, sizeof(DevState), hipMemcpyDeviceToHost) != hipSuccess) return HBF_EHIP;
  for (uint32_t k = 0; k < m->g.K; k++) h[0].die_free[k] = die_free[k] == INT64_MIN ? NEG : die_free[k];
  for (uint32_t c = 0; c < m->g.C; c++)
    h[0].chan_free[c] = chan_free[c] == INT64_MIN ? NEG : chan_free[c];
  if (hipMemcpy(m->st, h.data(), sizeof(DevState), hipMemcpyHostToDevice) != hipSuccess) return HBF_EHIP;
  return HBF_OK;
}

int hbf_profile(hbf_model_t m, int enable) {
  if (!m) return HBF_EINVAL;
  m->prof = enable != 0;
  m->prof_calls = 0;
  return HBF_OK;
}

int hbf_kernel_times(hbf_model_t m, float *ms, const char **names, int max, int *count) {
  if (!m || !count) return HBF_EINVAL;
  *count = 0;
  const int calls = std::min(m->prof_calls, hbf_model::RING);
  if (calls == 0) return HBF_OK;
  const int last = (m->prof_calls - 1) % hbf_model::RING;
  if (hipEventSynchronize(m->ev[last][kNumTimedKernels]) != hipSuccess) return HBF_EHIP;
  int k = 0;
  for (; k < kNumTimedKernels && k < max; k++) {
    double sum = 0.0;
    for (int c = 0; c < calls; c++) {
      float t = 0.f;
      if (hipEventElapsedTime(&t, m->ev[c][k], m->ev[c][k + 1]) != hipSuccess) return HBF_EHIP;
      sum += t;
    }
    if (ms) ms[k] = (float)(sum / calls);
    if (names) names[k] = kKernelNames[k];
  }
  *count = k;
  return HBF_OK;
}

const char *hbf_strerror(int code) {
  switch (code) {
    case HBF_OK: return "ok";
    case HBF_EINVAL: return "invalid argument";
    case HBF_EALIGN: return "range not page aligned";
    case HBF_EOVERLAP: return "range overlaps a registered range";
    case HBF_ENOWORKSPACE: return "workspace too small";
    case HBF_EUNSORTED: return "issue times decrease";
    case HBF_ERANGE_TIME: return "time outside the model's domain";
    case HBF_EHIP: return "HIP runtime error";
    case HBF_ENOMEM: return "out of memory";
    case HBF_EINTERNAL: return "internal wait bound exceeded";
    default: return "unknown status";
  }
}

}  // extern "C"
