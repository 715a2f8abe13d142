// Capacity-mode frame cache and next-page prefetcher (HBFSim, arXiv
// 2609.09800, Sections "D5: Capacity" and "D6: Speculative Prefetcher").
//
// A capacity range is served from a bounded frame cache in HBM: an access
// whose page is resident is a hit; otherwise it faults and its page is read
// from the media.  The prefetcher then reads ahead the pages after the
// faulting one.  Prefetch reads never enter the timing path, so this step
// only decides which accesses become media reads.  Reading: F frames with
// FIFO replacement (each insertion takes the frame filled longest ago; a hit
// changes nothing); a fault on page p inserts p and then, for k = 1..d in
// order while p + k < range_pages, each p + k not resident at that moment.
//
// The outcome of an access depends on every earlier one, so one wave runs
// one cache over the stream, 64 accesses per round; many caches -- a sweep
// over frame budgets and prefetch depths -- run as independent waves.
// Caches of up to CACHE_LDS_MAX frames keep their whole state in LDS;
// larger ones keep, in device memory, the number of each page's latest
// insertion (under FIFO, residency is a window over the insertion count).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

namespace {

__device__ __forceinline__ uint32_t lane_no() { return __lane_id(); }

// Device-memory accesses of the cache state, as global (not flat)
// instructions: a flat access also counts against the LDS wait counter, so
// every later LDS wait would wait for it too.
template <typename T>
using gptr = __attribute__((address_space(1))) T *;
template <typename T>
__device__ __forceinline__ T ld(const T *p) {
  return __hip_atomic_load((gptr<const T>)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st(T *p, T v) {
  __hip_atomic_store((gptr<T>)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
    if (c.frame_page) {
      c.frame_page[f] = -1;
      c.frame_pf[f] = 0;
    } else {
      c.fpf[f] = 0;
      c.fhit[f] = 0;
    }
  }
  if (c.pins)
    for (uint64_t q = t; q < R; q += stride) c.pins[q] = PINS_NEVER;
  if (t == 0) {
    c.ctl->head = 0;
    for (int k = 0; k < 5; k++) c.ctl->count[k] = 0;
    c.ctl->ins = 0;
    c.ctl->pend = 0;
  }
}

// ---- caches of more than CACHE_LDS_MAX frames: state in device memory
//
// With FIFO replacement the resident pages are exactly the last F pages
// inserted (a page is inserted only when absent, so those F are distinct):
// after I insertions, the page of insertion x is resident iff x >= I - F.
// The state is therefore the number of each page's latest insertion (pins,
// PINS_NEVER if none) and the counter I; insertion x fills frame x mod F,
// which keeps two flags (prefetched; hit since then), and eviction needs no
// bookkeeping of its own.  One wave runs one cache, 64 accesses per round:
//  - one gather of the pins of the round's pages; one of the candidates
//    (p+1 .. p+d) of the pages that miss at the start of the round; the
//    flags of the frames the round may refill, copied to LDS;
//  - the faults are then resolved in order inside the wave: a fault's
//    candidate k is inserted iff its latest insertion is below
//    I + c_k - F, with c_k the insertions of this fault before it (the
//    page itself first).  The condition is monotone in the set of
//    insertions, so iterating it from the candidates absent at the start
//    reaches the sequential answer in a few steps.  Later lanes and later
//    candidates see the round's insertions through a per-round list of
//    (page, first insertion, inserted-candidate mask);
//  - a page that becomes absent during the round (evicted by its own
//    round) loads its candidates when it faults.
// Evicting insertion x - F while inserting x counts a prefetched page
// evicted unused when its frame's flags say prefetched and not hit; the
// prefetched pages used are the prefetch reads minus those evicted unused
// minus those still resident and never hit (k_cache_pending).
constexpr int SNAP_CHUNK = 256;        // frame flags copied per chunk
constexpr int SNAP_MAX = 64 * 64;      // insertions in one round: 64 faults x (1 + 63 candidates)

// One wave runs one cache, and a wave's LDS operations execute in issue
// order, so between its own LDS writes and reads only the compiler must be
// kept from reordering or caching them (no wait is needed).
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

__global__ __launch_bounds__(64) void k_cache_run(const CacheCfg *__restrict__ cfgs, const int *cfg_ids, uint64_t R,
                                                  const uint64_t *__restrict__ pages, int64_t n,
                                                  uint8_t *__restrict__ hit, uint64_t *__restrict__ pf_page,
                                                  int64_t *__restrict__ pf_src, int64_t pf_cap,
                                                  const int64_t *status, int64_t *n_pf_out,
                                                  const ChunkCfg *__restrict__ ccfgs, int64_t i_base) {
  __shared__ int64_t s_cand[64 * 64];   // [slot][k]: latest insertion of candidate k of the slot-th start miss
  __shared__ int64_t s_page[64], s_cod[64];
  __shared__ uint32_t s_mlane[64];
  __shared__ int64_t s_fpm[64], s_fbase[64];
  __shared__ uint64_t s_fmask[64];
  __shared__ uint8_t s_snpf[SNAP_MAX], s_snhit[SNAP_MAX];
  __shared__ uint8_t s_ipf[SNAP_MAX], s_ihit[SNAP_MAX];  // the round's own insertions I_rs + u
  if (ld(status)) return;  // a page outside the range: nothing changes
  const int id = cfg_ids ? cfg_ids[blockIdx.x] : (int)blockIdx.x;
  if (ccfgs && ld(&ccfgs[id].ctl->valid)) return;  // this chunk was solved in parallel
  const CacheCfg c = cfgs[id];
  const uint32_t lane = lane_no(), d = c.d;
  const int64_t F = c.F;  // >= 64: an insertion offset within one fault (<= 63) is below F
  uint8_t *myhit = hit ? hit + (size_t)id * n : nullptr;
  const bool keep_pf = pf_page && id == 0;
  // state left by earlier launches: coherent loads, never the scalar cache
  int64_t I = ld(&c.ctl->ins);
  int64_t Imod = (int64_t)((uint64_t)I % (uint64_t)F);
  int64_t hits = 0, faults = 0, pfr = 0, unused_l = 0;
  int64_t npf = (id == 0 && n_pf_out) ? ld(n_pf_out) : 0;  // prefetch outputs of earlier chunks

  if (d == 0) {
    // No prefetch: a fault inserts only its own page, no frame is ever
    // prefetched, so only the insertion numbers matter.  Lane l of a round
    // faults iff no earlier lane of the round faulted on its page (such a
    // page stays resident for the rest of the round: a round inserts at most
    // 64 <= F pages) and its latest insertion is below I + c_l - F, with c_l
    // the faults of the lanes before it.  Each lane's outcome depends only
    // on those of the lanes before it, so the equations have one solution,
    // and iterating them from any guess reaches it after at most 64 steps
    // (after step k the first k lanes are settled); usually after 2.
    for (int64_t b0 = 0; b0 < n; b0 += 64) {
      const int64_t i = b0 + lane;
      const bool act = i < n;
      const uint32_t a = act ? (uint32_t)pages[i] : 0xFFFFFFFFu;
      const int64_t view = act ? ld(&c.pins[a]) : PINS_NEVER;
      // earlier lanes of the round with the same page
      uint64_t same = 0;
      for (uint32_t j = 0; j < 64; j++) {
        const uint32_t aj = (uint32_t)__builtin_amdgcn_readlane((int)a, (int)j);
        same |= (j < lane && aj == a) ? (1ull << j) : 0ull;
      }
      uint64_t fm = __ballot(act && view < I - F);
      for (int it = 0; it <= 64; it++) {
        const int64_t cl = (int64_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(fm >> 32),
                                                               __builtin_amdgcn_mbcnt_lo((uint32_t)fm, 0u));
        const uint64_t nf = __ballot(act && !(same & fm) && view < I + cl - F);
        if (nf == fm) break;
        fm = nf;
      }
      const bool flt = (fm >> lane) & 1;
      if (flt) {
        const int64_t cl = (int64_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(fm >> 32),
                                                               __builtin_amdgcn_mbcnt_lo((uint32_t)fm, 0u));
        st(&c.pins[a], I + cl);
      }
      if (act && myhit) myhit[i] = flt ? 0 : 1;
      const int64_t m = __popcll(fm);
      faults += m;
      hits += __popcll(__ballot(act)) - m;
      I += m;
    }
    if (lane == 0) {
      c.ctl->ins = I;
      c.ctl->head = (uint32_t)((uint64_t)I % (uint64_t)F);
      c.ctl->count[0] += hits;
      c.ctl->count[1] += faults;
      c.ctl->pend = 0;
    }
    return;
  }

  for (int64_t b0 = 0; b0 < n; b0 += 64) {
    const int64_t i = b0 + lane;
    const bool act = i < n;
    const int64_t a = act ? (int64_t)pages[i] : -1;
    int64_t view = act ? ld(&c.pins[a]) : PINS_NEVER;
    const int64_t I_rs = I, Imod_rs = Imod;
    // flags of the frames (Imod_rs + u) mod F, u < snap: they hold insertions
    // I_rs - F + u, which the round's insertions I_rs + u evict
    uint32_t snap = 0;
    auto load_snap = [&]() {
      uint8_t pf[SNAP_CHUNK / 64], hh[SNAP_CHUNK / 64];
#pragma unroll
      for (int u = 0; u < SNAP_CHUNK / 64; u++) {
        const int64_t fr = (int64_t)((uint32_t)(Imod_rs + (int64_t)(snap + u * 64 + lane)) % (uint32_t)F);
        pf[u] = ld(&c.fpf[fr]);
        hh[u] = ld(&c.fhit[fr]);
      }
#pragma unroll
      for (int u = 0; u < SNAP_CHUNK / 64; u++) {
        s_snpf[snap + u * 64 + lane] = pf[u];
        s_snhit[snap + u * 64 + lane] = hh[u];
      }
      snap += SNAP_CHUNK;
    };
    if (I_rs + 64 * (int64_t)(d + 1) > F) load_snap();  // the round may evict
    const uint64_t miss0 = __ballot(act && view < I_rs - F);
    int64_t fr = view >= 0 ? (int64_t)((uint64_t)view % (uint64_t)F) : 0;  // frame of this lane's page
    // candidates of the first pages missing at the start of the round, as
    // many as one 512-entry gather holds (the earliest misses are the
    // likeliest faults: later ones are often filled by an earlier fault's
    // prefetch); a fault beyond them reads its candidates when it happens
    const uint32_t n_pre = d > 0 ? min((uint32_t)__popcll(miss0), 512u / d) : 0u;
    if (n_pre > 0) {
      s_page[lane] = a;
      if ((miss0 >> lane) & 1) s_mlane[__builtin_amdgcn_mbcnt_hi((uint32_t)(miss0 >> 32),
                                       __builtin_amdgcn_mbcnt_lo((uint32_t)miss0, 0u))] = lane;
      lds_fence();
      const uint32_t total = n_pre * d;
      for (uint32_t e0 = 0; e0 < total; e0 += 512) {
        int64_t v[8];
        uint32_t at[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const uint32_t e = e0 + (uint32_t)u * 64 + lane;
          v[u] = PINS_NEVER;
          at[u] = 0xFFFFFFFFu;
          if (e < total) {
            const uint32_t sl = e / d, k = e - sl * d + 1;
            const int64_t q = s_page[s_mlane[sl]] + (int64_t)k;
            at[u] = sl * 64 + k;
            if ((uint64_t)q < R) v[u] = ld(&c.pins[q]);
          }
        }
#pragma unroll
        for (int u = 0; u < 8; u++)
          if (at[u] != 0xFFFFFFFFu) s_cand[at[u]] = v[u];
      }
      lds_fence();
    }

    uint32_t cursor = 0, J = 0;
    int64_t fmin = 0, fmax = 0;  // least and greatest faulting page of the round (with candidates)
    uint64_t hitmask = 0;
    while (true) {
      const bool later = act && lane >= cursor;
      const uint64_t mm = __ballot(later && view < I - F);
      const uint32_t f = mm ? (uint32_t)__builtin_ctzll(mm) : 64u;
      // the accesses before the next fault hit (their bookkeeping is done at
      // the end of the round: a lane's view no longer changes after its turn)
      const uint64_t hm = __ballot(later && lane < f);
      hitmask |= hm;
      hits += __popcll(hm);
      if (f == 64) break;
      faults++;
      const int64_t pm = read_lane(a, f);
      const int64_t im = b0 + f;
      // candidate k = lane (lane 0: the page itself)
      const bool cv = lane <= d && (uint64_t)(pm + (int64_t)lane) < R;
      int64_t L = PINS_NEVER;
      const uint32_t slot = (uint32_t)__popcll(miss0 & ((1ull << f) - 1));
      if (((miss0 >> f) & 1) && slot < n_pre) {
        if (lane >= 1 && cv) L = s_cand[slot * 64 + lane];
      } else {
        // not among the gathered misses: read the candidates now (through
        // LDS, so that only this branch waits for device memory)
        if (lane >= 1 && cv) s_cod[lane] = ld(&c.pins[pm + (int64_t)lane]);
        lds_fence();
        if (lane >= 1 && cv) L = s_cod[lane];
      }
      // an earlier fault of this round can have inserted pm + lane only if
      // its page lies in [pm + 1 - d, pm + d]
      const bool near = J > 0 && fmin <= pm + (int64_t)d && fmax + (int64_t)d >= pm + 1;
      if (near && lane >= 1 && cv) {
        for (int j = (int)J - 1; j >= 0; j--) {
          const int64_t off = pm + (int64_t)lane - s_fpm[j];
          if (off >= 0 && off <= (int64_t)d) {
            const uint64_t fm = s_fmask[j];
            if ((fm >> off) & 1) {
              L = s_fbase[j] + __popcll(fm & ((1ull << off) - 1));
              break;
            }
          }
        }
      }
      // insertions: the least fixed point of ins_k = (L_k < I + c_k - F);
      // the first guess takes c_k = 1, which is exact for depth 1
      uint64_t msk = __ballot(cv && (lane == 0 || L < I + 1 - F));
      while (d > 1) {
        const int64_t ck = (int64_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(msk >> 32),
                                                               __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
        const uint64_t m2 = __ballot(cv && (lane == 0 || L < I + ck - F));
        if (m2 == msk) break;
        msk = m2;
      }
      const uint32_t m = (uint32_t)__popcll(msk);
      // the flags of the frames these insertions take must be in the copy
      // before any later hit of this round could touch them (counted at the
      // end of the round)
      if (I + (int64_t)m > F) {
        int64_t need = I + (int64_t)m - I_rs;
        if (need > F) need = F;  // beyond F the evicted insertions are the round's own
        if ((int64_t)snap < need) {
          while ((int64_t)snap < need) load_snap();
          lds_fence();
        }
      }
      if ((msk >> lane) & 1) {
        const uint32_t off = __builtin_amdgcn_mbcnt_hi((uint32_t)(msk >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
        const int64_t x = I + off;
        int64_t fx = Imod + off;
        if (fx >= F) fx -= F;
        s_ipf[x - I_rs] = lane > 0 ? 1 : 0;
        s_ihit[x - I_rs] = 0;
        const int64_t q = pm + (int64_t)lane;
        st(&c.pins[q], x);
        st(&c.fpf[fx], (uint8_t)(lane > 0 ? 1 : 0));
        st(&c.fhit[fx], (uint8_t)0);
        if (lane > 0 && keep_pf) {
          const int64_t j = npf + (int64_t)off - 1;
          if (j < pf_cap) {
            pf_page[j] = (uint64_t)q;
            pf_src[j] = i_base + im;
          }
        }
      }
      npf += m - 1;
      pfr += m - 1;
      if (d > 0) {
        if (lane == 0) {
          s_fpm[J] = pm;
          s_fbase[J] = I;
          s_fmask[J] = msk;
        }
        fmin = J ? (pm < fmin ? pm : fmin) : pm;
        fmax = J ? (pm > fmax ? pm : fmax) : pm;
      }
      // the later accesses see this fault's insertions
      {
        const int64_t off = a - pm;
        if (act && lane > f && off >= 0 && off <= (int64_t)d && ((msk >> off) & 1)) {
          const int64_t o = __popcll(msk & ((1ull << off) - 1));
          view = I + o;
          fr = Imod + o;
          if (fr >= F) fr -= F;
        }
      }
      J++;
      I += m;
      Imod += m;
      if (Imod >= F) Imod -= F;
      wave_lds_order();
      cursor = f + 1;
    }
    const bool hl = (hitmask >> lane) & 1;
    if (act && myhit) myhit[i] = hl ? 1 : 0;
    if (hl) {
      // mark the hit insertion in the round's records or the flag copy, and
      // in device memory if it is still resident (else its frame was refilled)
      if (view >= I_rs) {
        s_ihit[view - I_rs] = 1;
      } else {
        const int64_t u = view - (I_rs - F);
        if (u >= 0 && u < (int64_t)snap) s_snhit[u] = 1;
      }
      if (view >= I - F) st(&c.fhit[fr], (uint8_t)1);
    }
    wave_lds_order();
    // evictions of the round: its insertions I_rs + u with I_rs + u >= F took
    // the frames of insertions I_rs - F + u -- made before the round (their
    // flags are in the copy) or, when u >= F, by the round itself (in its
    // own records); every hit on an evicted insertion preceded its eviction
    {
      const int64_t lo = F - I_rs > 0 ? F - I_rs : 0, hi = I - I_rs;
      for (int64_t u = lo + lane; u < hi; u += 64) {
        const bool gone_unused = u >= F ? (s_ipf[u - F] && !s_ihit[u - F]) : (s_snpf[u] && !s_snhit[u]);
        unused_l += gone_unused ? 1 : 0;
      }
    }
    lds_fence();
  }
  int64_t unused = unused_l;
  for (int o = 32; o >= 1; o >>= 1) unused += __shfl_xor(unused, o);
  if (lane == 0) {
    c.ctl->ins = I;
    c.ctl->head = (uint32_t)Imod;
    c.ctl->count[0] += hits;
    c.ctl->count[1] += faults;
    c.ctl->count[2] += pfr;
    c.ctl->count[4] += unused;
    c.ctl->pend = 0;
    if (id == 0 && n_pf_out) *n_pf_out = npf;
  }
}

// Prefetched pages still resident and never hit, per cache (after k_cache_run).
__global__ __launch_bounds__(256) void k_cache_pending(const CacheCfg *__restrict__ cfgs, const int *cfg_ids,
                                                      const int64_t *status) {
  __shared__ int64_t part[4];
  if (ld(status)) return;  // the run changed nothing
  const CacheCfg c = cfgs[cfg_ids ? cfg_ids[blockIdx.y] : (int)blockIdx.y];
  int64_t cnt = 0;
  for (uint64_t f = (uint64_t)blockIdx.x * 256 + threadIdx.x; f < c.F; f += (uint64_t)gridDim.x * 256)
    cnt += (c.fpf[f] && !c.fhit[f]) ? 1 : 0;
  for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t s = part[0] + part[1] + part[2] + part[3];
    if (s) atomicAdd((unsigned long long *)&c.ctl->pend, (unsigned long long)s);
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
  // device-memory caches: prefetched used = reads - evicted unused - still pending
  if (cfgs[b].pins) out[(size_t)b * per_cfg + 3] = ctl->count[2] - ctl->count[4] - ctl->pend;
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
  else {
    hipLaunchKernelGGL(k_cache_run, dim3((uint32_t)n_cfg), dim3(64), 0, s, dev_cfgs, cfg_ids, R, pages, n, hit,
                       pf_page, pf_src, pf_cap, status, n_pf_out, (const ChunkCfg *)nullptr, (int64_t)0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_cache_pending(dev_cfgs, cfg_ids, n_cfg, max_f, status, s);
  }
  return hipGetLastError();
}

hipError_t launch_cache_check(const uint64_t *pages, int64_t n, uint64_t R, int64_t *status, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cache_check, dim3((uint32_t)blocks), dim3(256), 0, s, pages, n, R, status);
  return hipGetLastError();
}

hipError_t launch_cache_pending(const CacheCfg *dev_cfgs, const int *cfg_ids, int n_cfg, uint32_t max_f,
                                const int64_t *status, hipStream_t s) {
  uint64_t pb = ((uint64_t)max_f + 255) / 256;
  if (pb > 256) pb = 256;
  hipLaunchKernelGGL(k_cache_pending, dim3((uint32_t)pb, (uint32_t)n_cfg), dim3(256), 0, s, dev_cfgs, cfg_ids, status);
  return hipGetLastError();
}

hipError_t launch_cache_seq(const CacheCfg *dev_cfgs, const ChunkCfg *dev_ccfgs, const int *cfg_ids, int n_cfg,
                            uint64_t R, const uint64_t *pages, int64_t n, int64_t i_base, uint8_t *hit,
                            uint64_t *pf_page, int64_t *pf_src, int64_t pf_cap, const int64_t *status,
                            int64_t *n_pf_out, hipStream_t s) {
  hipLaunchKernelGGL(k_cache_run, dim3((uint32_t)n_cfg), dim3(64), 0, s, dev_cfgs, cfg_ids, R, pages, n, hit,
                     pf_page, pf_src, pf_cap, status, n_pf_out, dev_ccfgs, i_base);
  return hipGetLastError();
}

}  // namespace hbf
