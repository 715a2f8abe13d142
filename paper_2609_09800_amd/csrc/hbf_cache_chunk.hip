// Chunked parallel solve of a device-memory frame cache (HBFSim, arXiv
// 2609.09800, Sections "D5: Capacity" and "D6: Speculative Prefetcher";
// FIFO replacement and next-page prefetch as read in hbf_cache.hip).
//
// Within one chunk of accesses, suppose first that nothing is evicted.  The
// resident set then only grows, so:
//  - an access can fault only as the first access of its page q in the
//    chunk, at time A(q), and only if q was not resident when the chunk
//    began (q is then a candidate);
//  - a candidate q faults iff no candidate q - k (1 <= k <= d) faulted at
//    an earlier time A(q - k) < A(q) (such a fault inserted q, or found it
//    resident).  Along the page axis this is a recurrence of width d: one
//    wave walks each segment of candidates (a gap of more than d pages
//    separates two segments), 64 pages at a time;
//  - page r is inserted at tau(r), the earliest fault among r - d .. r, if
//    it was not resident when the chunk began.  A fault's insertions are
//    numbered in page order after those of every earlier fault (a prefix
//    sum over the chunk's accesses).
// The answer is the true one iff every residency decision it took holds
// under FIFO: each page's last hit, and each prefetch candidate found
// resident, must still lie within the last F insertions at that moment.
// The check runs on the device; a chunk that passes is committed (hit
// flags, frame flags, evictions of prefetched pages never hit, counters),
// one that fails is undone and served by the sequential wave.  Nothing
// scales with the range: per-page state is tagged with the chunk's epoch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

namespace {

constexpr uint32_t NONE32 = 0xFFFFFFFFu;

template <typename T>
using gptr = __attribute__((address_space(1))) T *;
template <typename T>
__device__ __forceinline__ T ldr(const T *p) {
  return __hip_atomic_load((gptr<const T>)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ uint32_t rdl(uint32_t v, uint32_t l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)l);
}
__device__ __forceinline__ uint32_t ctz64(uint64_t m) { return (uint32_t)__builtin_ctzll(m); }
__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__popcll(m); }

// One append slot per set lane of `want` (wave-aggregated atomic).
__device__ __forceinline__ uint32_t wave_append(uint32_t *counter, bool want) {
  const uint64_t m = __ballot(want);
  uint32_t b = 0;
  if (lane_id() == 0 && m) b = atomicAdd(counter, popc(m));
  b = rdl(b, 0);
  return b + popc(m & ((1ull << lane_id()) - 1));
}

__device__ __forceinline__ int64_t wave_sum(int64_t v) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

struct Tags {
  uint64_t a, t;  // first access (~epoch), last access and insertion time (epoch)
  __device__ explicit Tags(uint32_t epoch) : a((uint64_t)(~epoch) << 32), t((uint64_t)epoch << 32) {}
};
constexpr uint64_t HI = 0xFFFFFFFF00000000ull;

}  // namespace

// Tags of the chunk's first and last access per page; counts cleared.
__global__ __launch_bounds__(256) void k_chunk_tag(const CacheCfg *__restrict__ cfgs, const ChunkCfg *__restrict__ ccs,
                                                   const int *ids, const uint64_t *__restrict__ pages, int64_t L,
                                                   uint32_t epoch, const int64_t *status, const int64_t *n_pf) {
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < L; j += (int64_t)gridDim.x * 256) {
    const uint64_t p = pages[j];
    atomicMin((unsigned long long *)&cc.at[p], (unsigned long long)(tg.a | (uint64_t)j));
    atomicMax((unsigned long long *)&cc.lt[p], (unsigned long long)(tg.t | (uint64_t)j));
    cc.S[j] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    cc.S[L] = 0;
    cc.ctl->nseg = 0;
    cc.ctl->valid = 1;
    cc.ctl->lost_old = 0;
    cc.ctl->I0 = ldr(&cfgs[id].ctl->ins);
    cfgs[id].ctl->pend = 0;  // recounted once the call's chunks have run
    cc.ctl->npf0 = (id == ids[0] && n_pf) ? ldr(n_pf) : 0;
  }
}

// Segment starts: candidates with no candidate among the d pages below.
__global__ __launch_bounds__(256) void k_chunk_starts(const CacheCfg *__restrict__ cfgs,
                                                      const ChunkCfg *__restrict__ ccs, const int *ids,
                                                      const uint64_t *__restrict__ pages, int64_t L, uint32_t epoch,
                                                      const int64_t *status) {
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const CacheCfg c = cfgs[id];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  const int64_t lim = ldr(&cc.ctl->I0) - (int64_t)c.F;  // resident at the start iff pins >= lim
  const int64_t span = ((L + 255) / 256) * 256;
  for (int64_t j0 = (int64_t)blockIdx.x * 256; j0 < span; j0 += (int64_t)gridDim.x * 256) {
    const int64_t j = j0 + threadIdx.x;
    bool start = false;
    uint64_t q_start = 0;
    if (j < L) {
      const uint64_t p = pages[j];
      if (cc.at[p] == (tg.a | (uint64_t)j) && c.pins[p] < lim) {
        start = true;
        for (uint32_t k = 1; k <= c.d && k <= p; k++) {
          const uint64_t q = p - k;
          if ((cc.at[q] & HI) == tg.a && c.pins[q] < lim) {
            start = false;
            break;
          }
        }
      }
      if (start) q_start = p;
    }
    const uint32_t k = wave_append(&cc.ctl->nseg, start);  // every lane of the wave, converged
    if (start && k < cc.Lmax) cc.seg[k] = (uint32_t)q_start;
  }
}

// One wave per segment: faults, insertion times, per-fault insertion
// counts and each insertion's rank within its fault, all written as plain
// stores (the tagged per-page word and the fault's count), so that the
// page state of the next four groups stays in flight while one is resolved.
namespace {
struct Walk {
  uint64_t lastc;   // last candidate of the segment so far
  uint32_t pa;      // previous group: this lane's first-access time
  uint64_t open;    // previous group: faults whose windows reach this group
  uint32_t pcnt;    // previous group: insertions so far of this lane's open fault
  uint32_t lastA;   // the largest first-access time among the segment's candidates so far
  bool hasA;
};

// Resolve the 64 pages at `base`; returns true once the segment has ended.
//
// Where the candidates' first-access times increase along the pages (a
// scan) and at most one fault reaches in from the previous group, every
// earlier fault within d pages blocks a candidate, so the faults are the
// greedy choice of candidates more than d pages apart, each page lies in
// at most one fault's window, and insertion time, rank and per-fault
// counts follow per lane.  Other groups take the general path: the lowest
// candidate not blocked by an earlier fault of smaller time is a fault.
__device__ __forceinline__ bool walk_group(Walk &w, uint64_t base, uint64_t at_c, int64_t pin_c, uint64_t R,
                                           uint32_t d, int64_t lim, const Tags &tg, const ChunkCfg &cc) {
  const uint32_t lane = lane_id();
  const uint64_t lt = (1ull << lane) - 1;
  const uint64_t le = lane == 63 ? ~0ull : (2ull << lane) - 1;
  const uint64_t r = base + lane;
  const bool inR = r < R;
  const uint32_t a = inR && (at_c & HI) == tg.a ? (uint32_t)at_c : NONE32;
  const bool nonres = inR && pin_c < lim;
  const bool cand = a != NONE32 && nonres;
  const uint64_t cm = __ballot(cand);
  // the segment continues while candidates are at most d pages apart
  const uint64_t below = cm & lt;
  const uint64_t prevpos = below ? base + 63 - (uint64_t)__builtin_clzll(below) : w.lastc;
  const uint64_t brk = __ballot(cand && r - prevpos > d);
  const uint64_t segc = brk ? (cm & ((1ull << ctz64(brk)) - 1)) : cm;
  if (segc) w.lastc = base + 63 - (uint64_t)__builtin_clzll(segc);
  const bool in_ext = inR && r <= w.lastc + d;
  const bool last = !(w.lastc + d >= base + 64 && base + 64 < R);
  // do the segment's candidates so far have increasing first-access times?
  const bool sc = (segc >> lane) & 1;
  const uint64_t sbelow = segc & lt;
  const uint32_t apl = (uint32_t)__shfl((int)a, sbelow ? 63 - __builtin_clzll(sbelow) : lane);
  const bool viol = sc && (sbelow ? apl >= a : (w.hasA && w.lastA >= a));
  const bool mono = !__ballot(viol) && popc(w.open) <= 1;

  uint64_t fm = 0, nopen = 0;
  uint32_t tau = NONE32, rank = 0, cnt = 0, ncnt = 0;
  bool fin_prev = false, fin_cur = false, ins = false;
  if (mono) {
    uint64_t rem = segc;
    const uint32_t g = w.open ? ctz64(w.open) : 0;
    if (w.open) rem &= ~((2ull << (g + d - 64)) - 1);  // lanes within the open fault's window
    while (rem) {
      const uint32_t f = ctz64(rem);
      fm |= 1ull << f;
      rem = f + d >= 63 ? 0 : rem & ~((2ull << (f + d)) - 1);
    }
    const uint64_t fb = fm & le;
    const uint32_t fs = fb ? 63 - __builtin_clzll(fb) : lane;
    const uint32_t af = (uint32_t)__shfl((int)a, fs);
    const bool cov = fb && lane - fs <= d;
    const uint32_t ag = w.open ? rdl(w.pa, g) : NONE32;
    const uint32_t c0 = w.open ? rdl(w.pcnt, g) : 0;
    const bool cov_prev = !cov && w.open && lane + 64 - g <= d;
    tau = cov ? af : (cov_prev ? ag : NONE32);
    ins = in_ext && tau != NONE32 && nonres;
    const uint64_t im = __ballot(ins);
    rank = cov ? popc(im & lt & ~((1ull << fs) - 1)) : c0 + popc(im & lt);
    if (w.open && lane == g) {
      fin_prev = true;
      ncnt = c0 + popc(im & ((2ull << (g + d - 64)) - 1));
    }
    if ((fm >> lane) & 1) {
      const uint64_t win = (lane + d >= 63 ? ~0ull : (2ull << (lane + d)) - 1) & ~lt;
      cnt = popc(im & win);
      fin_cur = lane + d < 64 || last;
    }
    nopen = __ballot(((fm >> lane) & 1) && !fin_cur);
  } else {
    uint64_t rem = segc;
    for (uint64_t m = w.open; m; m &= m - 1) {
      const uint32_t g = ctz64(m);
      const uint32_t ag = rdl(w.pa, g);
      rem &= ~__ballot(lane + 64 - g <= d && ag < a);
    }
    while (rem) {
      const uint32_t f = ctz64(rem);
      fm |= 1ull << f;
      const uint32_t af = rdl(a, f);
      rem &= ~(1ull << f);
      rem &= ~__ballot(lane > f && lane - f <= d && af < a);
    }
    // insertion time: the earliest fault whose window holds this page
    for (uint64_t m = w.open; m; m &= m - 1) {
      const uint32_t g = ctz64(m);
      const uint32_t ag = rdl(w.pa, g);
      if (lane + 64 - g <= d) tau = ag < tau ? ag : tau;
    }
    for (uint64_t m = fm; m; m &= m - 1) {
      const uint32_t f = ctz64(m);
      const uint32_t af = rdl(a, f);
      if (lane >= f && lane - f <= d) tau = af < tau ? af : tau;
    }
    ins = in_ext && tau != NONE32 && nonres;
    for (uint64_t m = w.open; m; m &= m - 1) {  // windows that end in this group
      const uint32_t g = ctz64(m);
      const uint32_t ag = rdl(w.pa, g);
      const bool mine = ins && tau == ag;
      const uint64_t mm = __ballot(mine);
      const uint32_t c0 = rdl(w.pcnt, g);
      if (mine) rank = c0 + popc(mm & lt);
      if (lane == g) {
        fin_prev = true;
        ncnt = c0 + popc(mm);  // the count of the previous group's fault in this lane
      }
    }
    for (uint64_t m = fm; m; m &= m - 1) {
      const uint32_t f = ctz64(m);
      const uint32_t af = rdl(a, f);
      const bool mine = ins && tau == af;
      const uint64_t mm = __ballot(mine);
      if (mine) rank = popc(mm & lt);
      if (lane == f) cnt = popc(mm);
      if (f + d < 64 || last) {
        if (lane == f) fin_cur = true;
      } else {
        nopen |= 1ull << f;
      }
    }
  }
  // the largest first-access time among the segment's candidates
  if (segc) {
    uint32_t mx = sc ? a : 0;
    if (mono) {
      mx = rdl(a, 63 - __builtin_clzll(segc));
    } else {
      for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t y = (uint32_t)__shfl_xor((int)mx, o);
        mx = y > mx ? y : mx;
      }
      mx = rdl(mx, 0);
    }
    w.lastA = w.hasA && w.lastA > mx ? w.lastA : mx;
    w.hasA = true;
  }
  // per-fault counts (packed: insertions << 32 | 1) and the page words
  if (fin_prev) cc.S[w.pa] = ((uint64_t)ncnt << 32) | 1u;
  if (fin_cur) cc.S[a] = ((uint64_t)cnt << 32) | 1u;
  if (ins) cc.tt[r] = tg.t | ((uint64_t)rank << 24) | tau;
  w.pa = a;
  w.open = nopen;
  w.pcnt = cnt;
  return last;
}
}  // namespace

__global__ __launch_bounds__(256) void k_chunk_walk(const CacheCfg *__restrict__ cfgs, const ChunkCfg *__restrict__ ccs,
                                                    const int *ids, uint64_t R, uint32_t epoch,
                                                    const int64_t *status) {
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const CacheCfg c = cfgs[id];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  const uint32_t lane = lane_id(), d = c.d;
  const int64_t lim = ldr(&cc.ctl->I0) - (int64_t)c.F;
  const uint32_t nseg_all = ldr(&cc.ctl->nseg);
  const uint32_t nseg = nseg_all < cc.Lmax ? nseg_all : cc.Lmax;
  // page state, loaded unconditionally (addresses clamped into the range;
  // lanes past the end are masked when the group is resolved)
  const gptr<const uint64_t> atg = (gptr<const uint64_t>)cc.at;
  const gptr<const int64_t> ping = (gptr<const int64_t>)c.pins;
  auto at_of = [&](uint64_t base) { return atg[base + lane < R ? base + lane : R - 1]; };
  auto pin_of = [&](uint64_t base) { return ping[base + lane < R ? base + lane : R - 1]; };
  for (uint32_t si = blockIdx.x * 4 + threadIdx.x / 64; si < nseg; si += gridDim.x * 4) {
    const uint64_t s = ldr(&cc.seg[si]);
    Walk w{s, NONE32, 0, 0, 0, false};
    // the next four groups in flight
    uint64_t a0 = at_of(s), a1 = at_of(s + 64), a2 = at_of(s + 128), a3 = at_of(s + 192);
    int64_t p0 = pin_of(s), p1 = pin_of(s + 64), p2 = pin_of(s + 128), p3 = pin_of(s + 192);
    for (uint64_t base = s;; base += 64) {
      const uint64_t at_c = a0;
      const int64_t pin_c = p0;
      a0 = a1;
      p0 = p1;
      a1 = a2;
      p1 = p2;
      a2 = a3;
      p2 = p3;
      a3 = at_of(base + 256);
      p3 = pin_of(base + 256);
      if (walk_group(w, base, at_c, pin_c, R, d, lim, tg, cc)) break;
    }
  }
}

// Exclusive scan of the packed per-access counts in two launches: the sum
// of each 1,024 accesses, then each block's scan offset by the sums before it.
namespace {
__device__ __forceinline__ uint64_t block_sum_1024(uint64_t v, uint64_t *part) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  if (lane_id() == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t t = 0;
  for (int w = 0; w < 16; w++) t += part[w];
  return t;
}
}  // namespace

__global__ __launch_bounds__(1024) void k_chunk_bsum(const ChunkCfg *__restrict__ ccs, const int *ids, int64_t L,
                                                     const int64_t *status) {
  __shared__ uint64_t part[16];
  if (ldr(status)) return;
  const ChunkCfg cc = ccs[ids[blockIdx.y]];
  const int64_t j = (int64_t)blockIdx.x * 1024 + threadIdx.x;
  const uint64_t t = block_sum_1024(j < L ? cc.S[j] : 0, part);
  if (threadIdx.x == 0) cc.bs[blockIdx.x] = t;
}

namespace {
// The page word of r, if the fault at access A inserted it: its rank, else -1.
__device__ __forceinline__ int owned_rank(uint64_t v, const Tags &tg, uint32_t A) {
  return (v & (HI | 0xFFFFFFull)) == (tg.t | A) ? (int)((v >> 24) & 63u) : -1;
}
}  // namespace

// Second scan pass: each block's exclusive scan offset by the sums before
// it; then each fault in the block (an access j whose page word names j
// itself, rank 0) numbers its insertions: I0 + insertions before j + rank.
__global__ __launch_bounds__(1024) void k_chunk_scan(const CacheCfg *__restrict__ cfgs,
                                                     const ChunkCfg *__restrict__ ccs, const int *ids,
                                                     const uint64_t *__restrict__ pages, int64_t L, uint64_t R,
                                                     uint32_t epoch, const int64_t *status) {
  __shared__ uint64_t part[16];
  __shared__ uint64_t s_pre;
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const CacheCfg c = cfgs[id];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  if (w == 0) {  // the sums of the blocks before this one
    uint64_t p = 0;
    for (uint32_t i = lane; i < blockIdx.x; i += 64) p += cc.bs[i];
    for (int o = 32; o >= 1; o >>= 1) p += __shfl_xor(p, o);
    if (lane == 0) s_pre = p;
  }
  const int64_t j = (int64_t)blockIdx.x * 1024 + threadIdx.x;
  const uint64_t v = j < L ? cc.S[j] : 0;
  uint64_t x = v;  // inclusive scan within the wave
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o);
    if (lane >= (uint32_t)o) x += y;
  }
  if (lane == 63) part[w] = x;
  __syncthreads();
  uint64_t off = s_pre;
  for (uint32_t i = 0; i < w; i++) off += part[i];
  if (j >= L) return;
  const uint64_t sj = off + x - v;
  cc.S[j] = sj;
  if (j == L - 1) cc.S[L] = off + x;
  if (v == 0) return;  // not a fault
  const uint64_t p = pages[j];
  const int64_t x0 = ldr(&cc.ctl->I0) + (int64_t)(sj >> 32);
  for (uint32_t k = 0; k <= c.d && p + k < R; k++) {
    const int rk = owned_rank(cc.tt[p + k], tg, (uint32_t)j);
    if (rk >= 0) c.pins[p + k] = x0 + rk;
  }
}

// The check: every page's last hit, and every prefetch candidate found
// resident, lies within the last F insertions at that moment.  Also, read
// before anything changes: frames filled before the chunk and evicted
// within it that hold a prefetched page never hit (a page resident at the
// start and accessed in the chunk was hit before its eviction).
__global__ __launch_bounds__(256) void k_chunk_check(const CacheCfg *__restrict__ cfgs,
                                                     const ChunkCfg *__restrict__ ccs, const int *ids,
                                                     const uint64_t *__restrict__ pages, int64_t L, uint64_t R,
                                                     uint32_t epoch, const int64_t *status) {
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const CacheCfg c = cfgs[id];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  const int64_t I0 = ldr(&cc.ctl->I0), F = c.F;
  const int64_t I1 = I0 + (int64_t)(ldr(&cc.S[L]) >> 32);
  const uint32_t nblk_a = (uint32_t)((L + 255) / 256);
  bool bad = false;
  int64_t lost = 0;
  if (blockIdx.x < nblk_a) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j < L) {
      const uint64_t p = pages[j];
      const bool fault = cc.tt[p] == (tg.t | (uint64_t)j);
      if (cc.lt[p] == (tg.t | (uint64_t)j) && !fault)  // the page's last access, a hit
        bad = c.pins[p] < I0 + (int64_t)(cc.S[j] >> 32) - F;
      if (fault) {  // the candidates this fault found resident
        const int64_t at_fault = I0 + (int64_t)(cc.S[j] >> 32) - F;
        int64_t before = 1;
        for (uint32_t k = 1; k <= c.d && p + k < R; k++) {
          const uint64_t q = p + k;
          if (owned_rank(cc.tt[q], tg, (uint32_t)j) >= 0) {
            before++;
          } else if (c.pins[q] < at_fault + before) {
            bad = true;
            break;
          }
        }
      } else if (cc.at[p] == (tg.a | (uint64_t)j)) {
        const int64_t x = c.pins[p];
        if (x >= I0 - F && x < I0 && x < I1 - F) {
          const uint64_t fr = (uint64_t)x % (uint64_t)F;
          lost -= (c.fpf[fr] && !c.fhit[fr]) ? 1 : 0;
        }
      }
    }
  } else {
    const int64_t ylo = I0 - F > 0 ? I0 - F : 0, yhi = I1 - F < I0 ? I1 - F : I0;
    for (int64_t y = ylo + (int64_t)(blockIdx.x - nblk_a) * 256 + threadIdx.x; y < yhi;
         y += (int64_t)(gridDim.x - nblk_a) * 256) {
      const uint64_t fr = (uint64_t)y % (uint64_t)F;
      lost += (c.fpf[fr] && !c.fhit[fr]) ? 1 : 0;
    }
  }
  if (__ballot(bad) && lane_id() == 0) cc.ctl->valid = 0;
  lost = wave_sum(lost);
  if (lane_id() == 0 && lost) atomicAdd((unsigned long long *)&cc.ctl->lost_old, (unsigned long long)lost);
}

// Commit, per access (checked chunks): hit flags; a hit on a page resident
// at the start marks its frame; each fault's insertions still resident set
// their frame flags, those evicted within the chunk count as unused when
// prefetched and never hit, prefetch outputs; then the counters.  A chunk
// that failed its check is undone instead, so that the sequential run
// starts from the chunk's initial state (a page not resident at the start
// stays so).  The frames written here are distinct: they hold the last F
// insertions.
__global__ __launch_bounds__(256) void k_chunk_commit(const CacheCfg *__restrict__ cfgs,
                                                      const ChunkCfg *__restrict__ ccs, const int *ids,
                                                      const uint64_t *__restrict__ pages, int64_t c0, int64_t L,
                                                      uint64_t R, uint32_t epoch, uint8_t *hit, uint64_t *pf_page,
                                                      int64_t *pf_src, int64_t pf_cap, const int64_t *status,
                                                      int64_t *n_pf) {
  if (ldr(status)) return;
  const int id = ids[blockIdx.y];
  const CacheCfg c = cfgs[id];
  const ChunkCfg cc = ccs[id];
  const Tags tg(epoch);
  const bool ok = ldr(&cc.ctl->valid) != 0;
  const uint64_t tot = ldr(&cc.S[L]);
  const int64_t I0 = ldr(&cc.ctl->I0), F = c.F, nf = (uint32_t)tot, M = (int64_t)(tot >> 32), I1 = I0 + M;
  const bool keep_pf = pf_page && id == ids[0];
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  int64_t lost = 0;
  if (j < L) {
    const uint64_t p = pages[j];
    const bool fault = cc.tt[p] == (tg.t | (uint64_t)j);
    if (ok && hit) hit[c0 + j] = fault ? 0 : 1;
    if (ok && !fault && cc.at[p] == (tg.a | (uint64_t)j)) {
      const int64_t x = c.pins[p];
      if (x >= I1 - F && x < I0) c.fhit[(uint64_t)x % (uint64_t)F] = 1;
    }
    if (fault) {
      const uint64_t sj = cc.S[j];
      const int64_t pf_before = ldr(&cc.ctl->npf0) + (int64_t)(sj >> 32) - (int64_t)(uint32_t)sj;
      for (uint32_t k = 0; k <= c.d && p + k < R; k++) {
        const uint64_t r = p + k;
        const int rk = owned_rank(cc.tt[r], tg, (uint32_t)j);
        if (rk < 0) continue;
        if (!ok) {
          c.pins[r] = PINS_NEVER;
          continue;
        }
        const int64_t x = c.pins[r];
        const uint64_t l = cc.lt[r];
        const bool used = (l & HI) == tg.t && (uint32_t)l > (uint32_t)j;
        if (x >= I1 - F) {
          const uint64_t fr = (uint64_t)x % (uint64_t)F;
          c.fpf[fr] = rk > 0 ? 1 : 0;
          c.fhit[fr] = used ? 1 : 0;
        } else {
          lost += (rk > 0 && !used) ? 1 : 0;
        }
        if (keep_pf && rk > 0) {
          const int64_t q = pf_before + rk - 1;
          if (q >= 0 && q < pf_cap) {
            pf_page[q] = r;
            pf_src[q] = c0 + j;
          }
        }
      }
    }
  }
  lost = wave_sum(lost);
  if (lane_id() == 0 && lost) atomicAdd((unsigned long long *)&c.ctl->count[4], (unsigned long long)lost);
  if (ok && blockIdx.x == 0 && threadIdx.x == 0) {
    c.ctl->count[0] += L - nf;
    c.ctl->count[1] += nf;
    c.ctl->count[2] += M - nf;
    atomicAdd((unsigned long long *)&c.ctl->count[4], (unsigned long long)ldr(&cc.ctl->lost_old));
    c.ctl->ins = I1;
    c.ctl->head = (uint32_t)((uint64_t)I1 % (uint64_t)F);
    if (keep_pf && n_pf) *n_pf = ldr(&cc.ctl->npf0) + M - nf;
  }
}

__global__ __launch_bounds__(256) void k_chunk_clear(const ChunkCfg *__restrict__ ccs, const int *ids, uint64_t R) {
  const ChunkCfg cc = ccs[ids[blockIdx.y]];
  for (uint64_t q = (uint64_t)blockIdx.x * 256 + threadIdx.x; q < R; q += (uint64_t)gridDim.x * 256) {
    cc.at[q] = ~0ull;
    cc.lt[q] = 0;
    cc.tt[q] = 0;
  }
}

hipError_t launch_chunk_clear(const ChunkCfg *dev_ccfgs, const int *cfg_ids, int n_cfg, uint64_t R, hipStream_t s) {
  uint64_t b = (R + 255) / 256;
  if (b > 2048) b = 2048;
  hipLaunchKernelGGL(k_chunk_clear, dim3((uint32_t)b, (uint32_t)n_cfg), dim3(256), 0, s, dev_ccfgs, cfg_ids, R);
  return hipGetLastError();
}

hipError_t launch_cache_chunk(const CacheCfg *cfgs, const ChunkCfg *ccs, const int *ids, int n_cfg, uint32_t max_f,
                              uint32_t max_d, uint64_t R, const uint64_t *pages, int64_t c0, int64_t L,
                              uint32_t epoch, uint8_t *hit, uint64_t *pf_page, int64_t *pf_src, int64_t pf_cap,
                              int64_t *status, int64_t *n_pf, hipStream_t s) {
  (void)max_f;
  (void)max_d;
  const uint64_t *pg = pages + c0;
  const uint32_t nb = (uint32_t)((L + 255) / 256);
  const uint32_t nsb = (uint32_t)((L + 1023) / 1024);
  const uint32_t walk = nb < 1024 ? nb : 1024;  // 4 waves per block, one segment each at a time
  const uint32_t nev = 256;                     // blocks over the evictions of earlier frames
  hipLaunchKernelGGL(k_chunk_tag, dim3(nb, n_cfg), dim3(256), 0, s, cfgs, ccs, ids, pg, L, epoch, status, n_pf);
  hipLaunchKernelGGL(k_chunk_starts, dim3(nb, n_cfg), dim3(256), 0, s, cfgs, ccs, ids, pg, L, epoch, status);
  hipLaunchKernelGGL(k_chunk_walk, dim3(walk, n_cfg), dim3(256), 0, s, cfgs, ccs, ids, R, epoch, status);
  hipLaunchKernelGGL(k_chunk_bsum, dim3(nsb, n_cfg), dim3(1024), 0, s, ccs, ids, L, status);
  hipLaunchKernelGGL(k_chunk_scan, dim3(nsb, n_cfg), dim3(1024), 0, s, cfgs, ccs, ids, pg, L, R, epoch, status);
  hipLaunchKernelGGL(k_chunk_check, dim3(nb + nev, n_cfg), dim3(256), 0, s, cfgs, ccs, ids, pg, L, R, epoch,
                     status);
  hipLaunchKernelGGL(k_chunk_commit, dim3(nb, n_cfg), dim3(256), 0, s, cfgs, ccs, ids, pg, c0, L, R, epoch, hit,
                     pf_page, pf_src, pf_cap, status, n_pf);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_cache_seq(cfgs, ccs, ids, n_cfg, R, pg, L, c0, hit ? hit + c0 : nullptr, pf_page, pf_src, pf_cap,
                          status, n_pf, s);
}

}  // namespace hbf
