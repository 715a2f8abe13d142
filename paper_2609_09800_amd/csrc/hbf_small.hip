// Small calls in one launch (HBFSim, arXiv 2609.09800, Section "Design": the
// online media model, a die-read queue then a channel-transfer queue, each
// FCFS).  A call of at most one chunk (4,096 requests) is otherwise bound
// by its dozen launches, not by its work.  Here one workgroup does it all:
//   1. classify and validate, and rank each request among the chunk's
//      requests of its die queue (stable: index order);
//   2. stage the chunk in die order (queue-major) and take the Lindley form
//      of each die queue as one segmented prefix maximum:
//      die_done_r = (r+1)*tR + max(L, max over i <= r of issue_i - i*tR);
//   3. place each request in its channel's service order: its rank there is
//      the number of the channel's requests, over all of its die runs
//      (each sorted by die-done), that come before it by (die-done, index),
//      found by a binary search per run;
//   4. the channel's Lindley form, again as one segmented prefix maximum:
//      complete_r = (r+1)*xfer + max(F, max over i <= r of die_done_i - i*xfer);
//   5. new clocks, or, on any error, HBF_TIME_ERROR everywhere and the clocks
//      left as they were.
// It serves the plain two-stage model (no refresh quanta pending, no
// register blocking, not the vmem route) with at most SMALL_K die queues, at
// most SMALL_DK per channel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_device.h"
#include "hbf_internal.h"

namespace hbf {

namespace {

DEVI size_t up16(size_t x) { return (x + 15) & ~size_t(15); }

// LDS: ranges | wcnt[DWAVES][K] u16 | tot[K] u16 | seg[K+1] u32 | cf[C] i64 |
//      sdd[CHUNK] i64 | cdd[CHUNK] i64 | sidx, skey, cidx, cch [CHUNK] u16
struct SmallLayout {
  size_t wcnt, tot, seg, cf, sdd, cdd, sidx, skey, cidx, cch, total;
};
__host__ __device__ inline SmallLayout small_layout(uint32_t K, uint32_t C) {
  SmallLayout L;
  size_t o = (sizeof(LdsRanges) + 15) & ~size_t(15);
  L.wcnt = o; o += (size_t)DWAVES * K * 2;
  L.tot = o;  o += (size_t)K * 2;
  o = (o + 15) & ~size_t(15);
  L.seg = o;  o += (size_t)(K + 1) * 4;
  o = (o + 15) & ~size_t(15);
  L.cf = o;   o += (size_t)C * 8;
  L.sdd = o;  o += (size_t)CHUNK * 8;
  L.cdd = o;  o += (size_t)CHUNK * 8;
  L.sidx = o; o += (size_t)CHUNK * 2;
  L.skey = o; o += (size_t)CHUNK * 2;
  L.cidx = o; o += (size_t)CHUNK * 2;
  L.cch = o;  o += (size_t)CHUNK * 2;
  L.total = o;
  return L;
}


// Stable rank of each item among this wave's items with the same key (item,
// then lane order), and the wave's per-key counts in wcnt.  The lanes that
// share a key are found with one ballot per key bit (a small call's keys
// are few, so many lanes of a wave share one).
DEVI void wave_rank_bits(const uint32_t *key, uint32_t *rank, uint16_t *wcnt, uint32_t nbits) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int e = 0; e < DITEMS; e++) {
    const uint32_t k = key[e];
    const bool valid = k != KEY_NONE;
    uint64_t mask = __ballot(valid);
    for (uint32_t b = 0; b < nbits; b++) {
      const bool bit = (k >> b) & 1u;
      const uint64_t bb = __ballot(valid && bit);
      mask &= bit ? bb : ~bb;
    }
    const uint32_t below = mask_below(mask), cnt = (uint32_t)__popcll(mask);
    uint32_t prior = 0;
    if (valid) prior = wcnt[k];
    // all reads of this item happen before the group's first lane updates
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (valid && below == 0) wcnt[k] = (uint16_t)(prior + cnt);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    rank[e] = prior + below;
  }
}

}  // namespace

template <bool POW2>
__global__ __launch_bounds__(DBLK) void k_small(const uint64_t *__restrict__ addr, const int64_t *__restrict__ issue,
                                               int64_t n, int64_t *__restrict__ complete, Geo g, RangeTable rt,
                                               DevState *st, CallCtl *ctl) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ uint32_t shsum[DWAVES];
  __shared__ SegMax shseg[DWAVES];
  __shared__ uint32_t s_err, s_maxrun;
  __shared__ int64_t s_max;
  const uint32_t K = g.K, Dk = g.Dk, C = g.C;
  const SmallLayout SL = small_layout(K, C);
  LdsRanges *lr = (LdsRanges *)smem;
  uint16_t *wcnt = (uint16_t *)(smem + SL.wcnt);
  uint16_t *tot = (uint16_t *)(smem + SL.tot);
  uint32_t *seg = (uint32_t *)(smem + SL.seg);
  int64_t *cf = (int64_t *)(smem + SL.cf);
  int64_t *sdd = (int64_t *)(smem + SL.sdd);
  int64_t *cdd = (int64_t *)(smem + SL.cdd);
  uint16_t *sidx = (uint16_t *)(smem + SL.sidx);
  uint16_t *skey = (uint16_t *)(smem + SL.skey);
  uint16_t *cidx = (uint16_t *)(smem + SL.cidx);
  uint16_t *cch = (uint16_t *)(smem + SL.cch);
  const uint32_t t = threadIdx.x, lane = lane_id(), w = t >> 6;
  const int64_t tR = g.tR, xfer = g.xfer;

  load_ranges(lr, rt);
  for (uint32_t q = t; q < DWAVES * K; q += DBLK) wcnt[q] = 0;
  if (t == 0) {
    s_err = 0;
    s_maxrun = 0;
    s_max = NEG;
  }
  __syncthreads();
  const RangeReg rr = range_reg(lr);
  uint32_t errb = 0;

  // 1. classify, validate, rank within the die queue (item e of wave w:
  //    requests w*512 + e*64 + lane)
  const int64_t wb = (int64_t)w * 64 * DITEMS;
  uint32_t key[DITEMS], rank[DITEMS];
  int64_t iss[DITEMS];
#pragma unroll
  for (int e = 0; e < DITEMS; e++) {
    const int64_t i = wb + e * 64 + lane;
    const bool v = i < n;
    const int64_t x = v ? issue[i] : 0;
    uint32_t k = KEY_NONE;
    if (v) {
      if (x < 0 || x >= ISSUE_LIMIT) errb |= ERR_RANGE_TIME;
      if (i > 0 && x < issue[i - 1]) errb |= ERR_UNSORTED;
      k = key_of<POW2>(g, lr, rr, addr[i]);
      if (k == KEY_NONE) complete[i] = x;  // native path: no modeled delay
    }
    key[e] = k;
    iss[e] = x;
  }
  uint32_t nbits = 0;
  while ((1u << nbits) < K) nbits++;
  wave_rank_bits(key, rank, wcnt + w * K, nbits);
  __syncthreads();
  cross_wave_offsets(wcnt, tot, K);
  __syncthreads();
  {  // each queue's run in die order
    const uint32_t per = (K + DBLK - 1) / DBLK;
    const uint32_t a0 = t * per, b0 = min(K, a0 + per);
    uint32_t sum = 0;
    for (uint32_t k = a0; k < b0; k++) sum += tot[k];
    uint32_t ex;
    const uint32_t all = block_excl_sum<DWAVES>(sum, &ex, shsum);
    for (uint32_t k = a0; k < b0; k++) {
      seg[k] = ex;
      ex += tot[k];
    }
    if (t == 0) seg[K] = all;
    uint32_t longest = 0;
    for (uint32_t k = a0; k < b0; k++) longest = max(longest, (uint32_t)tot[k]);
    if (longest) atomicMax(&s_maxrun, longest);
  }
  __syncthreads();
  // 2. stage issue_r - r*tR in die order; a run's head also takes the die clock
#pragma unroll
  for (int e = 0; e < DITEMS; e++) {
    const uint32_t k = key[e];
    if (k != KEY_NONE) {
      const uint32_t rc = wcnt[w * K + k] + rank[e];
      const uint32_t P = seg[k] + rc;
      int64_t v = iss[e] - (int64_t)rc * tR;
      if (rc == 0) v = imax(v, st->die_free[k]);
      sdd[P] = v;
      sidx[P] = (uint16_t)(wb + e * 64 + lane);
      skey[P] = (uint16_t)k;
    }
  }
  __syncthreads();
  const uint32_t m = seg[K];
  const uint32_t p0 = t * DITEMS;
  {
    int64_t vals[DITEMS];
    SegMax agg = {0, NEG};
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      const uint32_t p = p0 + q;
      vals[q] = NEG;
      if (p < m) {
        vals[q] = sdd[p];
        agg = seg_comb(agg, SegMax{p == seg[skey[p]], vals[q]});
      }
    }
    const SegMax ex = block_excl_segmax<DWAVES>(agg, shseg);
    int64_t run = ex.v;
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      const uint32_t p = p0 + q;
      if (p < m) {
        const uint32_t r = p - seg[skey[p]];
        run = r == 0 ? vals[q] : imax(run, vals[q]);
        const int64_t dd = (int64_t)(r + 1) * tR + run;
        if (dd >= TIME_LIMIT) errb |= ERR_OVERFLOW;
        sdd[p] = dd;
      }
    }
  }
  __syncthreads();
  // 3. channel service order.  A request's rank in its channel counts, in
  // each die run of the channel, the entries before it (its own run: its
  // position).  A thread's requests are consecutive in die order, mostly of
  // one run, so their counts in another run only grow: the first is found by
  // a binary search, the next ones by walking on from the previous count.
  {
    uint32_t top = 1;  // the largest power of two not above the longest run
    while (2 * top <= CHUNK && 2 * top <= (uint32_t)s_maxrun) top *= 2;
    uint32_t kq[DITEMS], r[DITEMS];
    int64_t dq[DITEMS];
    uint32_t iq[DITEMS];
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      const uint32_t p = p0 + q;
      kq[q] = KEY_NONE;
      r[q] = 0;
      dq[q] = 0;
      iq[q] = 0;
      if (p < m) {
        kq[q] = skey[p];
        dq[q] = sdd[p];
        iq[q] = sidx[p];
      }
    }
    // entry j of the staged order comes before (d0, i0)
    auto before = [&](uint32_t j, int64_t d0, uint32_t i0) {
      const int64_t v = sdd[j];
      const uint32_t sv = sidx[j];
      return (v < d0) | ((v == d0) & (sv < i0));
    };
    for (uint32_t d = 0; d < Dk; d++) {
      uint32_t prev_key = KEY_NONE, cnt = 0;
#pragma unroll
      for (int q = 0; q < DITEMS; q++) {
        if (kq[q] != KEY_NONE) {
          const uint32_t kk = (kq[q] / Dk) * Dk + d;
          if (kk == kq[q]) {
            r[q] += p0 + q - seg[kk];  // its own run: its position
          } else {
            const uint32_t lo = seg[kk], len = tot[kk];
            if (kq[q] != prev_key) {  // the thread's first request of this run: binary search
              cnt = 0;
              for (uint32_t step = top; step > 0; step >>= 1) {
                const uint32_t at = cnt + step;
                if (at <= len && before(lo + at - 1, dq[q], iq[q])) cnt = at;
              }
            } else {
              while (cnt < len && before(lo + cnt, dq[q], iq[q])) cnt++;
            }
            r[q] += cnt;
          }
          prev_key = kq[q];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      if (kq[q] != KEY_NONE) {
        const uint32_t c = kq[q] / Dk;
        const uint32_t cp = seg[c * Dk] + r[q];
        cdd[cp] = dq[q];
        cidx[cp] = (uint16_t)iq[q];
        cch[cp] = (uint16_t)c;
      }
    }
  }
  __syncthreads();
  // 4. channel completions; a channel's head also takes the channel clock
  {
    int64_t vals[DITEMS];
    SegMax agg = {0, NEG};
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      const uint32_t p = p0 + q;
      vals[q] = NEG;
      if (p < m) {
        const uint32_t c = cch[p], h = seg[c * Dk];
        int64_t v = cdd[p] - (int64_t)(p - h) * xfer;
        if (p == h) v = imax(v, st->chan_free[c]);
        vals[q] = v;
        agg = seg_comb(agg, SegMax{p == h, v});
      }
    }
    const SegMax ex = block_excl_segmax<DWAVES>(agg, shseg);
    int64_t run = ex.v, mx = NEG;
#pragma unroll
    for (int q = 0; q < DITEMS; q++) {
      const uint32_t p = p0 + q;
      if (p < m) {
        const uint32_t c = cch[p], h = seg[c * Dk];
        run = p == h ? vals[q] : imax(run, vals[q]);
        const int64_t cpl = (int64_t)(p - h + 1) * xfer + run;
        if (cpl >= TIME_LIMIT) errb |= ERR_OVERFLOW;
        complete[cidx[p]] = cpl;
        mx = imax(mx, cpl);
        if (p + 1 == seg[(c + 1) * Dk]) cf[c] = cpl;  // the channel's last
      }
    }
    if (mx > NEG) atomicMax((long long *)&s_max, (long long)mx);
  }
  if (errb) atomicOr(&s_err, errb);
  __syncthreads();
  // 5. clocks, or the failure
  const uint32_t err = s_err;
  if (err) {
    for (int64_t i = t; i < n; i += DBLK) complete[i] = HBF_TIME_ERROR;
    if (t == 0) {
      atomicOr(&st->sticky, err);
      ctl->err = err;
      ctl->n_in = m;
      ctl->max_cpl = NEG;
    }
    return;
  }
  for (uint32_t k = t; k < K; k += DBLK)
    if (tot[k]) st->die_free[k] = sdd[seg[k] + tot[k] - 1];
  for (uint32_t c = t; c < C; c += DBLK)
    if (seg[(c + 1) * Dk] > seg[c * Dk]) st->chan_free[c] = cf[c];
  if (t == 0) {
    ctl->err = 0;
    ctl->n_in = m;
    ctl->max_cpl = s_max;
  }
}

bool small_path_ok(const Geo &g, int64_t n, bool refresh) {
  return !refresh && !g.reg_block && !g.vmem && n > 0 && n <= CHUNK && g.K <= SMALL_K && g.Dk <= SMALL_DK &&
         small_layout(g.K, g.C).total <= SMALL_LDS_MAX;
}

size_t lds_small(const Geo &g) { return small_layout(g.K, g.C).total; }

hipError_t launch_small(const Geo &g, const RangeTable &rt, DevState *st, CallCtl *ctl, const uint64_t *addr,
                        const int64_t *issue, int64_t n, int64_t *complete, hipStream_t s) {
  const size_t lds = lds_small(g);
  if (g.pow2)
    hipLaunchKernelGGL(k_small<true>, dim3(1), dim3(DBLK), lds, s, addr, issue, n, complete, g, rt, st, ctl);
  else
    hipLaunchKernelGGL(k_small<false>, dim3(1), dim3(DBLK), lds, s, addr, issue, n, complete, g, rt, st, ctl);
  return hipGetLastError();
}

// (the largest LDS any geometry on this path asks for)
hipError_t set_lds_small() {
  const int lds = SMALL_LDS_MAX;
  hipError_t e = hipFuncSetAttribute((const void *)k_small<true>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void *)k_small<false>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}

}  // namespace hbf
