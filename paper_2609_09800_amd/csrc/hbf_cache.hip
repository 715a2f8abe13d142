// Capacity-mode frame cache and next-page prefetcher (HBFSim, arXiv
// 2609.09800, Sections "D5: Capacity" and "D6: Speculative Prefetcher").
//
// A capacity range is served from a bounded frame cache in HBM: an access
// whose page is resident is a hit; otherwise it faults and its page is read
// from the media.  The prefetcher then fetches the pages that follow the
// faulting page.  Prefetch reads never enter the timing path, so this step
// only decides which accesses become media reads.  Reading: F frames with
// FIFO replacement (each insertion takes the frame filled longest ago; a hit
// changes nothing); a fault on page p inserts p and then, for k = 1..d in
// order while p + k < range_pages, each p + k not resident at that moment.
//
// The outcome of an access depends on every earlier one, so one wave runs
// one cache over the stream.  It takes the accesses 64 at a time: all 64
// look their pages up at once; every access before the first fault is a
// hit (hits change nothing); the fault's insertions are done by up to d+1
// lanes at once (FIFO slots are head, head+1, ...); the accesses after it
// look up again.  A fault whose insertion would evict one of its own later
// candidates (which was resident when the fault began) is replayed by one
// lane in order.  Many caches -- a sweep over frame budgets and prefetch
// depths -- run as independent waves.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

namespace {

__device__ __forceinline__ uint32_t lane_no() { return __lane_id(); }

template <typename T>
__device__ __forceinline__ T ld(const T *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st(T *p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t take_flag(uint32_t *p) {
  return __hip_atomic_exchange(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wave_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
  __builtin_amdgcn_wave_barrier();
}
__device__ __forceinline__ int64_t read_lane(int64_t v, uint32_t l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, (int)l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), (int)l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

}  // namespace

// Page check: status = HBF_EINVAL if any page lies outside the range.
__global__ __launch_bounds__(256) void k_cache_check(const uint64_t *__restrict__ pages, int64_t n, uint64_t R,
                                                     int64_t *status) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    bad |= pages[i] >= R;
  if (__ballot(bad) && lane_no() == 0) atomicExch((unsigned long long *)status, (unsigned long long)HBF_EINVAL);
}

__global__ __launch_bounds__(256) void k_cache_clear(CacheCfg *cfgs, uint64_t R) {
  const CacheCfg c = cfgs[blockIdx.y];
  const uint64_t t = (uint64_t)blockIdx.x * 256 + threadIdx.x, stride = (uint64_t)gridDim.x * 256;
  for (uint64_t f = t; f < c.F; f += stride) {
    c.frame_page[f] = -1;
    c.frame_pf[f] = 0;
  }
  if (c.slot)
    for (uint64_t q = t; q < R; q += stride) c.slot[q] = -1;
  if (t == 0) {
    c.ctl->head = 0;
    for (int k = 0; k < 5; k++) c.ctl->count[k] = 0;
  }
}

// One wave per cache (cache cfg_ids[blockIdx.x], or blockIdx.x).  hit:
// per-access flags of cache b at hit + b * n (nullable); the prefetch list
// (nullable) is kept for cache 0.
__global__ __launch_bounds__(64) void k_cache_run(const CacheCfg *__restrict__ cfgs, const int *cfg_ids, uint64_t R,
                                                  const uint64_t *__restrict__ pages, int64_t n,
                                                  uint8_t *__restrict__ hit, uint64_t *__restrict__ pf_page,
                                                  int64_t *__restrict__ pf_src, int64_t pf_cap,
                                                  const int64_t *status, int64_t *n_pf_out) {
  if (ld(status)) return;  // a page outside the range: nothing changes
  const int id = cfg_ids ? cfg_ids[blockIdx.x] : (int)blockIdx.x;
  const CacheCfg c = cfgs[id];
  const uint32_t lane = lane_no(), F = c.F, d = c.d;
  uint8_t *myhit = hit ? hit + (size_t)id * n : nullptr;
  const bool keep_pf = pf_page && id == 0;
  uint32_t head = c.ctl->head;
  int64_t hits = 0, faults = 0, pfr = 0, used = 0, unused = 0, npf = 0;

  for (int64_t b0 = 0; b0 < n; b0 += 64) {
    const int64_t i = b0 + lane;
    const int64_t p = i < n ? (int64_t)pages[i] : 0;
    uint64_t active = __ballot(i < n);
    while (active) {
      const bool act = (active >> lane) & 1;
      const int32_t s = act ? ld(&c.slot[p]) : -1;
      const uint64_t miss = __ballot(act && s < 0);
      const uint32_t f = miss ? (uint32_t)__builtin_ctzll(miss) : 64u;
      // accesses before the first fault hit the current contents
      const bool h = act && lane < f;
      bool first_use = false;
      if (h) {
        if (myhit) myhit[i] = 1;
        first_use = take_flag(&c.frame_pf[s]) != 0;
      }
      hits += __popcll(__ballot(h));
      used += __popcll(__ballot(first_use));
      if (f == 64) break;
      // the fault at lane f: candidates p_f + k, k = lane = 0..d
      const int64_t pm = read_lane(p, f);
      const int64_t im = b0 + f;
      if (lane == f && myhit) myhit[i] = 0;
      faults++;
      const int64_t cand = pm + (int64_t)lane;
      const bool cv = lane <= d && (uint64_t)cand < R;
      const bool res = cv && lane > 0 && ld(&c.slot[cand]) >= 0;
      const bool ins = cv && !res;
      const uint64_t insm = __ballot(ins);
      const uint32_t pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(insm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)insm, 0u));
      const uint32_t m = (uint32_t)__popcll(insm);
      const uint32_t fs = (uint32_t)(((uint64_t)head + pos) % F);
      const int64_t ev = ins ? ld(&c.frame_page[fs]) : -1;
      // does this insertion evict a later candidate that was resident (it
      // would have to be fetched again when its turn comes)?
      const int64_t k = ev - pm;
      const bool later = ins && k > (int64_t)lane && k <= (int64_t)d;
      const uint32_t kk = later ? (uint32_t)k : lane;
      const bool kres = __shfl(res ? 1 : 0, (int)kk) != 0;
      if (__ballot(later && kres)) {
        // replay this fault in order on one lane
        if (lane == 0) {
          for (uint32_t j = 0; j <= d && (uint64_t)(pm + j) < R; j++) {
            const int64_t q = pm + j;
            if (j > 0 && ld(&c.slot[q]) >= 0) continue;
            const int64_t old = ld(&c.frame_page[head]);
            if (old >= 0) {
              st(&c.slot[old], -1);
              if (take_flag(&c.frame_pf[head])) unused++;
            }
            st(&c.frame_page[head], q);
            st(&c.frame_pf[head], j > 0 ? 1u : 0u);
            st(&c.slot[q], (int32_t)head);
            if (j > 0) {
              if (keep_pf && npf < pf_cap) {
                pf_page[npf] = (uint64_t)q;
                pf_src[npf] = im;
              }
              npf++;
              pfr++;
            }
            head = head + 1 == F ? 0 : head + 1;
          }
        }
        head = (uint32_t)__shfl((int)head, 0);
        npf = read_lane(npf, 0);
        pfr = read_lane(pfr, 0);
        unused = read_lane(unused, 0);
      } else {
        bool lost = false;
        if (ins) {
          if (ev >= 0) {
            st(&c.slot[ev], -1);
            lost = take_flag(&c.frame_pf[fs]) != 0;
          }
          st(&c.frame_page[fs], cand);
          st(&c.frame_pf[fs], lane > 0 ? 1u : 0u);
          st(&c.slot[cand], (int32_t)fs);
          if (lane > 0 && keep_pf) {
            const int64_t j = npf + (int64_t)pos - 1;
            if (j < pf_cap) {
              pf_page[j] = (uint64_t)cand;
              pf_src[j] = im;
            }
          }
        }
        unused += __popcll(__ballot(lost));
        npf += m - 1;
        pfr += m - 1;
        head = (uint32_t)(((uint64_t)head + m) % F);
      }
      wave_fence();
      active &= ~((f == 63 ? ~0ull : ((1ull << (f + 1)) - 1)));
    }
  }
  if (lane == 0) {
    c.ctl->head = head;
    c.ctl->count[0] += hits;
    c.ctl->count[1] += faults;
    c.ctl->count[2] += pfr;
    c.ctl->count[3] += used;
    c.ctl->count[4] += unused;
    if (id == 0 && n_pf_out) *n_pf_out = npf;
  }
}

// ---- the same cache with its whole state in LDS (frames <= CACHE_LDS_MAX)
//
// LDS: fpage[F] (page per frame, -1 empty) | fpf[F] (prefetched, not hit
// yet) | tab[T]: open-addressed hash of the resident pages, linear probing,
// each 64-bit entry holding (page << 32 | frame), or EMPTY / TOMB (deleted)
// in the page half.  T is a power of two >= 4F (>= 2F at the largest F);
// the table is rebuilt when tombstones reach T/8, so probes stay short.
// Within a 64-access round, the accesses after a fault do not look their
// pages up again: each lane updates its page's residency from the fault's
// insertions and evictions in registers.

namespace {
constexpr uint32_t PG_EMPTY = 0xFFFFFFFFu;
constexpr uint32_t PG_TOMB = 0xFFFFFFFEu;
constexpr uint64_t ENT_EMPTY = ~0ull;

__device__ __forceinline__ uint64_t ent(uint32_t page, uint32_t frame) { return (uint64_t)page << 32 | frame; }

struct LdsCache {
  int32_t *fpage;
  uint32_t *fpf;
  uint64_t *tab;
  uint32_t tmask, tshift;
  __device__ uint32_t home(uint32_t p) const { return (p * 0x9E3779B1u) >> tshift; }
  // Probes are bounded by one pass over the table: a present key is met
  // within it, and an absent one is absent.
  __device__ int32_t find(uint32_t p) const {  // frame holding p, or -1
    uint32_t e = home(p);
    for (uint32_t t = 0; t <= tmask; t++, e = (e + 1) & tmask) {
      const uint64_t v = tab[e];
      const uint32_t pg = (uint32_t)(v >> 32);
      if (pg == p) return (int32_t)(uint32_t)v;
      if (pg == PG_EMPTY) return -1;
    }
    return -1;
  }
  __device__ void erase(uint32_t p, uint32_t f) {  // the entry (p, f) becomes a tombstone
    const uint64_t want = ent(p, f);
    uint32_t e = home(p);
    for (uint32_t t = 0; t <= tmask; t++, e = (e + 1) & tmask)
      if (tab[e] == want) {
        tab[e] = ent(PG_TOMB, 0);
        return;
      }
  }
  // Returns whether it reused a tombstone.  At most F entries are live, so a
  // free entry always remains; two passes bound the probing under contention.
  __device__ bool insert(uint32_t p, uint32_t f) {
    uint32_t e = home(p);
    for (uint32_t t = 0; t <= 2 * tmask + 1; t++, e = (e + 1) & tmask) {
      const uint64_t cur = tab[e];
      const uint32_t pg = (uint32_t)(cur >> 32);
      if ((pg == PG_EMPTY || pg == PG_TOMB) &&
          atomicCAS((unsigned long long *)&tab[e], (unsigned long long)cur, (unsigned long long)ent(p, f)) == cur)
        return pg == PG_TOMB;
    }
    return false;
  }
};

__device__ __forceinline__ void lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
}  // namespace

static __host__ __device__ uint32_t cache_tab_size(uint32_t F) {
  uint32_t T = 2;
  while (T < 4 * F) T <<= 1;
  if ((size_t)F * 8 + (size_t)T * 8 > 96 * 1024) T >>= 1;   // the largest caches: >= 2F
  return T;
}

__global__ __launch_bounds__(64) void k_cache_run_lds(const CacheCfg *__restrict__ cfgs, const int *cfg_ids,
                                                      uint64_t R, const uint64_t *__restrict__ pages, int64_t n,
                                                      uint8_t *__restrict__ hit, uint64_t *__restrict__ pf_page,
                                                      int64_t *__restrict__ pf_src, int64_t pf_cap,
                                                      const int64_t *status, int64_t *n_pf_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  if (ld(status)) return;  // a page outside the range: nothing changes
  const int id = cfg_ids ? cfg_ids[blockIdx.x] : (int)blockIdx.x;
  const CacheCfg c = cfgs[id];
  const uint32_t lane = lane_no(), F = c.F, d = c.d;
  uint8_t *myhit = hit ? hit + (size_t)id * n : nullptr;
  const bool keep_pf = pf_page && id == 0;
  const uint32_t T = cache_tab_size(F);
  LdsCache L;
  L.tab = (uint64_t *)smem;
  L.fpage = (int32_t *)(L.tab + T);
  L.fpf = (uint32_t *)(L.fpage + F);
  L.tmask = T - 1;
  L.tshift = 32 - (uint32_t)__builtin_ctz(T);
  // load the cache, then hash its resident pages
  for (uint32_t f = lane; f < F; f += 64) {
    L.fpage[f] = (int32_t)c.frame_page[f];
    L.fpf[f] = c.frame_pf[f];
  }
  for (uint32_t e = lane; e < T; e += 64) L.tab[e] = ENT_EMPTY;
  lds_fence();
  for (uint32_t f = lane; f < F; f += 64)
    if (L.fpage[f] >= 0) L.insert((uint32_t)L.fpage[f], f);
  lds_fence();
  uint32_t head = c.ctl->head;
  uint32_t tombs = 0;
  int64_t hits = 0, faults = 0, pfr = 0, used = 0, unused = 0, npf = 0;
  auto rebuild = [&]() {  // wave-uniform
    for (uint32_t e = lane; e < T; e += 64) L.tab[e] = ENT_EMPTY;
    lds_fence();
    for (uint32_t fr = lane; fr < F; fr += 64)
      if (L.fpage[fr] >= 0) L.insert((uint32_t)L.fpage[fr], fr);
    lds_fence();
    tombs = 0;
  };

  for (int64_t b0 = 0; b0 < n; b0 += 64) {
    const int64_t i = b0 + lane;
    const uint32_t p = i < n ? (uint32_t)pages[i] : 0u;
    uint64_t active = __ballot(i < n);
    int32_t s = (i < n) ? L.find(p) : -1;   // the frame holding p (kept current below)
    while (active) {
      const bool act = (active >> lane) & 1;
      const uint64_t miss = __ballot(act && s < 0);
      const uint32_t f = miss ? (uint32_t)__builtin_ctzll(miss) : 64u;
      const bool h = act && lane < f;   // before the first fault: hits
      bool first_use = false;
      if (h) {
        if (myhit) myhit[i] = 1;
        first_use = atomicExch(&L.fpf[s], 0u) != 0;
      }
      hits += __popcll(__ballot(h));
      used += __popcll(__ballot(first_use));
      if (f == 64) break;
      const uint32_t pm = (uint32_t)__builtin_amdgcn_readlane((int)p, (int)f);
      const int64_t im = b0 + f;
      if (lane == f && myhit) myhit[i] = 0;
      faults++;
      const uint32_t cand = pm + lane;
      const bool cv = lane <= d && (uint64_t)cand < R;
      // candidates' residency and the frames they would take, in one round
      const bool res = cv && lane > 0 && L.find(cand) >= 0;
      const uint32_t vs = (uint32_t)(((uint64_t)head + lane) % F);
      const int32_t vpage = lane <= d ? L.fpage[vs] : -1;   // page in the lane-th oldest frame
      const bool ins = cv && !res;
      const uint64_t insm = __ballot(ins);
      const uint32_t pos =
          __builtin_amdgcn_mbcnt_hi((uint32_t)(insm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)insm, 0u));
      const uint32_t m = (uint32_t)__popcll(insm);
      const uint32_t fs = (uint32_t)(((uint64_t)head + pos) % F);
      const int32_t ev = (int32_t)__shfl((int)vpage, (int)pos);  // page evicted by this lane's insertion
      const int64_t k = ins ? (int64_t)ev - (int64_t)pm : -1;
      const bool later = ins && ev >= 0 && k > (int64_t)lane && k <= (int64_t)d;
      const uint32_t kk = later ? (uint32_t)k : lane;
      const bool kres = __shfl(res ? 1 : 0, (int)kk) != 0;
      const uint32_t head0 = head;
      if (__ballot(later && kres)) {
        // an insertion would evict one of this fault's own later candidates:
        // replay the fault in order on one lane
        if (lane == 0) {
          for (uint32_t j = 0; j <= d && (uint64_t)pm + j < R; j++) {
            const uint32_t q = pm + j;
            if (j > 0 && L.find(q) >= 0) continue;
            const int32_t old = L.fpage[head];
            if (old >= 0) {
              L.erase((uint32_t)old, head);
              tombs++;
              if (L.fpf[head]) unused++;
            }
            L.fpage[head] = (int32_t)q;
            L.fpf[head] = j > 0 ? 1u : 0u;
            if (L.insert(q, head)) tombs--;
            if (j > 0) {
              if (keep_pf && npf < pf_cap) {
                pf_page[npf] = (uint64_t)q;
                pf_src[npf] = im;
              }
              npf++;
              pfr++;
            }
            head = head + 1 == F ? 0 : head + 1;
          }
        }
        head = (uint32_t)__shfl((int)head, 0);
        tombs = (uint32_t)__shfl((int)tombs, 0);
        npf = read_lane(npf, 0);
        pfr = read_lane(pfr, 0);
        unused = read_lane(unused, 0);
        lds_fence();
        if (tombs * 8 >= T) rebuild();
        active &= ~((f == 63 ? ~0ull : ((1ull << (f + 1)) - 1)));
        s = ((active >> lane) & 1) ? L.find(p) : -1;   // look up again after a replay
        continue;
      }
      // evictions first, then the new pages
      bool lost = false;
      if (ins && ev >= 0) {
        L.erase((uint32_t)ev, fs);
        lost = L.fpf[fs] != 0;
      }
      tombs += (uint32_t)__popcll(__ballot(ins && ev >= 0));
      unused += __popcll(__ballot(lost));
      lds_fence();
      if (ins) {
        L.fpage[fs] = (int32_t)cand;
        L.fpf[fs] = lane > 0 ? 1u : 0u;
      }
      lds_fence();
      const bool reused = ins && L.insert(cand, fs);
      tombs -= (uint32_t)__popcll(__ballot(reused));
      if (ins && lane > 0 && keep_pf) {
        const int64_t j = npf + (int64_t)pos - 1;
        if (j < pf_cap) {
          pf_page[j] = (uint64_t)cand;
          pf_src[j] = im;
        }
      }
      npf += m - 1;
      pfr += m - 1;
      head = (uint32_t)(((uint64_t)head0 + m) % F);
      lds_fence();
      // the accesses still to come update their page's frame in registers:
      // a page among the fault's candidates that was inserted now sits in
      // that candidate's frame; a page whose frame was taken is gone
      active &= ~((f == 63 ? ~0ull : ((1ull << (f + 1)) - 1)));
      {
        const uint32_t off = p - pm;                       // candidate slot of this lane's page
        const bool in_c = p >= pm && off <= d && (uint64_t)p < R;
        const uint32_t src = in_c ? off : lane;
        const bool c_ins = __shfl(ins ? 1 : 0, (int)src) != 0;
        const uint32_t c_fs = (uint32_t)__shfl((int)fs, (int)src);
        const uint32_t rel = (uint32_t)(((uint64_t)(s >= 0 ? (uint32_t)s : 0u) + F - head0) % F);
        if (in_c && c_ins)
          s = (int32_t)c_fs;
        else if (s >= 0 && rel < m)
          s = -1;
      }
      if (tombs * 8 >= T) rebuild();
    }
  }
  // write the cache back
  for (uint32_t fr = lane; fr < F; fr += 64) {
    c.frame_page[fr] = L.fpage[fr];
    c.frame_pf[fr] = L.fpf[fr];
  }
  if (lane == 0) {
    c.ctl->head = head;
    c.ctl->count[0] += hits;
    c.ctl->count[1] += faults;
    c.ctl->count[2] += pfr;
    c.ctl->count[3] += used;
    c.ctl->count[4] += unused;
    if (id == 0 && n_pf_out) *n_pf_out = npf;
  }
}

static size_t cache_lds_bytes(uint32_t F) { return (size_t)cache_tab_size(F) * 8 + (size_t)F * 8; }

hipError_t cache_set_lds_limit() {
  return hipFuncSetAttribute((const void *)k_cache_run_lds, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)cache_lds_bytes(CACHE_LDS_MAX));
}

// Copy the counters out: per cache `per_cfg` int64 = the five counters,
// then (when per_cfg >= 7) this call's prefetch reads and status.
__global__ void k_cache_report(const CacheCfg *__restrict__ cfgs, int n_cfg, const int64_t *n_pf,
                               const int64_t *status, int64_t *out, int per_cfg) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= n_cfg) return;
  const CacheCtl *ctl = cfgs[b].ctl;
  for (int k = 0; k < 5; k++) out[(size_t)b * per_cfg + k] = ctl->count[k];
  if (per_cfg >= 7) {
    out[(size_t)b * per_cfg + 5] = n_pf ? *n_pf : 0;
    out[(size_t)b * per_cfg + 6] = *status;
    for (int k = 7; k < per_cfg; k++) out[(size_t)b * per_cfg + k] = 0;
  }
}

hipError_t launch_cache_report(const CacheCfg *dev_cfgs, int n_cfg, const int64_t *n_pf, const int64_t *status,
                               int64_t *out, int per_cfg, hipStream_t s) {
  hipLaunchKernelGGL(k_cache_report, dim3((n_cfg + 63) / 64), dim3(64), 0, s, dev_cfgs, n_cfg, n_pf, status, out,
                     per_cfg);
  return hipGetLastError();
}

hipError_t launch_cache_clear(CacheCfg *dev_cfgs, int n_cfg, uint64_t R, uint32_t max_f, hipStream_t s) {
  uint64_t w = R > max_f ? R : max_f;
  uint64_t blocks = (w + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cache_clear, dim3((uint32_t)blocks, (uint32_t)n_cfg), dim3(256), 0, s, dev_cfgs, R);
  return hipGetLastError();
}

hipError_t launch_cache_run(const CacheCfg *dev_cfgs, const int *cfg_ids, int n_cfg, bool lds, uint32_t max_f,
                            uint64_t R, const uint64_t *pages, int64_t n, uint8_t *hit, uint64_t *pf_page,
                            int64_t *pf_src, int64_t pf_cap, int64_t *status, int64_t *n_pf_out, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cache_check, dim3((uint32_t)blocks), dim3(256), 0, s, pages, n, R, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (lds)
    hipLaunchKernelGGL(k_cache_run_lds, dim3((uint32_t)n_cfg), dim3(64), cache_lds_bytes(max_f), s, dev_cfgs,
                       cfg_ids, R, pages, n, hit, pf_page, pf_src, pf_cap, status, n_pf_out);
  else
    hipLaunchKernelGGL(k_cache_run, dim3((uint32_t)n_cfg), dim3(64), 0, s, dev_cfgs, cfg_ids, R, pages, n, hit,
                       pf_page, pf_src, pf_cap, status, n_pf_out);
  return hipGetLastError();
}

}  // namespace hbf
