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
  for (uint64_t q = t; q < R; q += stride) c.slot[q] = -1;
  if (t == 0) {
    c.ctl->head = 0;
    for (int k = 0; k < 5; k++) c.ctl->count[k] = 0;
  }
}

// One wave per cache (blockIdx.x).  hit: per-access flags of cache b at
// hit + b * n (nullable); the prefetch list (nullable) is kept for cache 0.
__global__ __launch_bounds__(64) void k_cache_run(const CacheCfg *__restrict__ cfgs, uint64_t R,
                                                  const uint64_t *__restrict__ pages, int64_t n,
                                                  uint8_t *__restrict__ hit, uint64_t *__restrict__ pf_page,
                                                  int64_t *__restrict__ pf_src, int64_t pf_cap,
                                                  const int64_t *status, int64_t *n_pf_out) {
  if (ld(status)) return;  // a page outside the range: nothing changes
  const CacheCfg c = cfgs[blockIdx.x];
  const uint32_t lane = lane_no(), F = c.F, d = c.d;
  uint8_t *myhit = hit ? hit + (size_t)blockIdx.x * n : nullptr;
  const bool keep_pf = pf_page && blockIdx.x == 0;
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
    if (blockIdx.x == 0 && n_pf_out) *n_pf_out = npf;
  }
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

hipError_t launch_cache_run(const CacheCfg *dev_cfgs, int n_cfg, uint64_t R, const uint64_t *pages, int64_t n,
                            uint8_t *hit, uint64_t *pf_page, int64_t *pf_src, int64_t pf_cap, int64_t *status,
                            int64_t *n_pf_out, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cache_check, dim3((uint32_t)blocks), dim3(256), 0, s, pages, n, R, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_cache_run, dim3((uint32_t)n_cfg), dim3(64), 0, s, dev_cfgs, R, pages, n, hit, pf_page,
                     pf_src, pf_cap, status, n_pf_out);
  return hipGetLastError();
}

}  // namespace hbf
