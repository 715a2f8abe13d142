// HIP kernels (gfx950, wave64) of the HBF service-model hot path.
//
// hbf_time_requests computes, for every request, the completion of a
// die-read queue followed by a channel-transfer queue (the online media
// model of HBFSim, arXiv 2609.09800, Section "Design"; the two-stage reading
// of that model is documented in hbf.h).  Each stage is a first-come
// first-served single server with a constant service time S, whose
// departures obey the Lindley form
//
//     f_m = m*S + max(f_0, max_{i<=m} (a_i - (i-1)*S))          (m = 1, 2, ...)
//
// for arrivals a_1 <= ... in service order and a server free at f_0.  Both
// stages are therefore a rank computation plus a prefix maximum, done here
// with exact int64 arithmetic:
//
//   k_die_reduce   pass 1 over the requests: classify + map (Section D1),
//                  validate issue times, write complete = issue for the
//                  native path, and per (tile, die queue) the count and the
//                  departure of the tile's last request from an idle die.
//   k_tile_scan    per die queue, compose the tiles in order -> each tile's
//                  incoming die clock and rank offset; new die clocks.
//   k_key_scan     die-queue segment offsets; the time-cell grid.
//   k_die_scatter  pass 2: exact die-done times, written in die-queue order
//                  (an LDS-staged stable multisplit) plus, per (channel,
//                  time cell, die), the first die rank in that cell.
//   k_channel_merge per (channel, time cell): merge the cell's die runs in
//                  LDS by (die-done, index), prefix-max, chain the channel
//                  clock across cells with a decoupled look-back, scatter
//                  complete[] in request order.
//   k_finalize     fail-closed error fill, or commit of the new clocks.
//
// A die emits at most one request per t_read_ns, so a time cell of width
// 2^shift <= T * t_read_ns holds at most T requests per die: cells are
// bounded by construction and need no sort of 64-bit keys.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

#define DEVI __device__ __forceinline__

DEVI int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }
DEVI int64_t imin(int64_t a, int64_t b) { return a < b ? a : b; }

DEVI uint32_t lane_id() { return __lane_id(); }

// number of lanes below this one whose bit is set in `mask`
DEVI uint32_t mask_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

DEVI uint64_t agent_load(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEVI void agent_store(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEVI uint32_t agent_load32(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// look-back status words: 0 = not yet published, else value + 2^62
DEVI uint64_t enc_time(int64_t x) { return (uint64_t)x + (uint64_t(1) << 62); }
DEVI int64_t dec_time(uint64_t w) { return (int64_t)(w - (uint64_t(1) << 62)); }

// ------------------------------------------------------------------ block scans

// Exclusive prefix sum over the block (256 threads); returns the block total.
DEVI uint32_t block_excl_sum(uint32_t v, uint32_t *excl, uint32_t *sh /*[WAVES]*/) {
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t y = __shfl_up(x, d);
    if (lane >= (uint32_t)d) x += y;
  }
  if (lane == 63) sh[w] = x;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < WAVES; i++) {
    uint32_t t = sh[i];
    base += (i < (int)w) ? t : 0u;
    tot += t;
  }
  __syncthreads();
  *excl = base + x - v;
  return tot;
}

// Exclusive prefix max over the block; identity NEG.
DEVI int64_t block_excl_max(int64_t v, int64_t *sh /*[WAVES]*/) {
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    int64_t y = __shfl_up(x, d);
    if (lane >= (uint32_t)d) x = imax(x, y);
  }
  if (lane == 63) sh[w] = x;
  int64_t ex = __shfl_up(x, 1);
  if (lane == 0) ex = NEG;
  __syncthreads();
  int64_t pre = NEG;
#pragma unroll
  for (int i = 0; i < WAVES; i++)
    if (i < (int)w) pre = imax(pre, sh[i]);
  __syncthreads();
  return imax(pre, ex);
}

// Exclusive segmented prefix max: element = (head flag, value).
struct SegMax {
  int f;
  int64_t v;
};
DEVI SegMax seg_comb(SegMax a, SegMax b) {
  SegMax r;
  r.f = a.f | b.f;
  r.v = b.f ? b.v : imax(a.v, b.v);
  return r;
}
DEVI SegMax block_excl_segmax(SegMax v, SegMax *sh /*[WAVES]*/) {
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  SegMax x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    SegMax y;
    y.f = __shfl_up(x.f, d);
    y.v = __shfl_up(x.v, d);
    if (lane >= (uint32_t)d) x = seg_comb(y, x);
  }
  if (lane == 63) sh[w] = x;
  SegMax ex;
  ex.f = __shfl_up(x.f, 1);
  ex.v = __shfl_up(x.v, 1);
  if (lane == 0) {
    ex.f = 0;
    ex.v = NEG;
  }
  __syncthreads();
  SegMax pre = {0, NEG};
#pragma unroll
  for (int i = 0; i < WAVES; i++)
    if (i < (int)w) pre = seg_comb(pre, sh[i]);
  __syncthreads();
  return seg_comb(pre, ex);
}

// ------------------------------------------------------------------ classification

// Copy the range table into LDS (dynamic indexing then stays in LDS).
struct LdsRanges {
  uint64_t base[MAX_RANGES];
  uint64_t bytes[MAX_RANGES];
  uint64_t pbase[MAX_RANGES];
  uint32_t rid[MAX_RANGES];
  int32_t n;
};

DEVI void load_ranges(LdsRanges *lr, const RangeTable &rt) {
  const int t = threadIdx.x;
  if (t < MAX_RANGES) {
    lr->base[t] = rt.base[t];
    lr->bytes[t] = rt.bytes[t];
    lr->pbase[t] = rt.pbase[t];
    lr->rid[t] = rt.rid[t];
  }
  if (t == 0) lr->n = rt.n;
}

// Index (in the sorted snapshot) of the range holding `a`, or -1.
DEVI int find_range(const LdsRanges *lr, uint64_t a) {
  int lo = 0, hi = lr->n;  // first range with base > a
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (lr->base[mid] <= a) lo = mid + 1;
    else hi = mid;
  }
  int r = lo - 1;
  if (r < 0) return -1;
  return (a - lr->base[r] < lr->bytes[r]) ? r : -1;
}

struct Loc {
  uint32_t ch, die, plane;
  uint64_t page;
};

// Device page -> (channel, die, plane, page), channel-first striping.
template <bool POW2>
DEVI Loc map_page(const Geo &g, uint64_t dp) {
  Loc L;
  if (POW2) {
    L.ch = (uint32_t)(dp & (g.C - 1));
    L.die = (uint32_t)((dp >> g.lg_C) & (g.D - 1));
    L.plane = (uint32_t)((dp >> (g.lg_C + g.lg_D)) & (g.P - 1));
    L.page = dp >> (g.lg_C + g.lg_D + g.lg_P);
  } else {
    uint64_t q = dp / g.C;
    L.ch = (uint32_t)(dp - q * g.C);
    uint64_t q2 = q / g.D;
    L.die = (uint32_t)(q - q2 * g.D);
    uint64_t q3 = q2 / g.P;
    L.plane = (uint32_t)(q2 - q3 * g.P);
    L.page = q3;
  }
  return L;
}

template <bool POW2>
DEVI uint64_t dev_page(const Geo &g, const LdsRanges *lr, int r, uint64_t a) {
  uint64_t off = a - lr->base[r];
  return lr->pbase[r] + (POW2 ? (off >> g.lg_page) : off / g.page_bytes);
}

// Die-queue key of an address, or KEY_NONE for the native path.
template <bool POW2>
DEVI uint32_t key_of(const Geo &g, const LdsRanges *lr, uint64_t a) {
  int r = find_range(lr, a);
  if (r < 0) return KEY_NONE;
  Loc L = map_page<POW2>(g, dev_page<POW2>(g, lr, r, a));
  uint32_t k = L.ch * g.D + L.die;
  if (g.plane_parallel) k = k * g.P + L.plane;
  return k;
}

// ------------------------------------------------------------------ die stage, shared

// Stable rank of each item among this wave's items with the same key, in
// (item, lane) order; wcnt is the wave's private per-key counter row.
// Match-any over the key bits: lanes whose keys agree on every bit are peers.
DEVI void wave_rank(const uint32_t *key, uint32_t *rank, uint16_t *wcnt, uint32_t kbits) {
#pragma unroll
  for (int e = 0; e < ITEMS; e++) {
    const uint32_t k = key[e];
    const bool valid = k != KEY_NONE;
    uint64_t peers = __ballot(valid);
    for (uint32_t b = 0; b < kbits; b++) {
      const bool bit = (k >> b) & 1u;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    uint32_t below = mask_below(peers);
    uint32_t prior = 0;
    if (valid) prior = wcnt[k];
    // all reads of this item happen before the leaders' writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (valid && below == 0) wcnt[k] = (uint16_t)(prior + __popcll(peers));
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    rank[e] = prior + below;
  }
}

// After wave_rank: turn wcnt[w][k] into the wave's exclusive offset among
// the block's waves and write the chunk total of key k to tot[k].
DEVI void cross_wave_offsets(uint16_t *wcnt, uint16_t *tot, uint32_t K) {
  for (uint32_t k = threadIdx.x; k < K; k += BLK) {
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < WAVES; w++) {
      uint32_t c = wcnt[w * K + k];
      wcnt[w * K + k] = (uint16_t)run;
      run += c;
    }
    tot[k] = (uint16_t)run;
  }
}

// ------------------------------------------------------------------ k_prologue

__global__ void k_prologue(CallCtl *ctl, uint64_t *st_agg, uint64_t *st_incl, size_t nst) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctl->err = 0;
    ctl->ticket = 0;
    ctl->n_in = 0;
    ctl->G = 0;
    ctl->shift = 0;
    ctl->max_dd = NEG;
    ctl->cbase = 0;
  }
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nst;
       i += (size_t)gridDim.x * blockDim.x) {
    st_agg[i] = 0;
    st_incl[i] = 0;
  }
}

// ------------------------------------------------------------------ k_die_reduce

// LDS: ranges | wcnt[WAVES][K] u16 | tot[K] u16 | cnt[K] u32 | amax[K] i64
template <bool POW2>
__global__ __launch_bounds__(BLK) void k_die_reduce(const uint64_t *__restrict__ addr,
                                                    const int64_t *__restrict__ issue, int64_t n,
                                                    int64_t *__restrict__ complete, Geo g,
                                                    RangeTable rt, int64_t tile_elems,
                                                    uint32_t *__restrict__ agg_cnt,
                                                    int64_t *__restrict__ agg_A, CallCtl *ctl,
                                                    uint32_t kbits) {
  extern __shared__ __align__(16) unsigned char smem[];
  LdsRanges *lr = (LdsRanges *)smem;
  const uint32_t K = g.K;
  int64_t *amax = (int64_t *)(smem + ((sizeof(LdsRanges) + 15) & ~size_t(15)));
  uint32_t *cnt = (uint32_t *)(amax + K);
  uint16_t *wcnt = (uint16_t *)(cnt + K);
  uint16_t *tot = wcnt + WAVES * K;

  load_ranges(lr, rt);
  for (uint32_t k = threadIdx.x; k < K; k += BLK) {
    cnt[k] = 0;
    amax[k] = NEG;
  }
  __syncthreads();

  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * tile_elems;
  const int64_t t1 = imin(n, t0 + tile_elems);
  const int64_t tR = g.tR;
  uint32_t errb = 0;
  uint16_t *mycnt = wcnt + w * K;

  for (int64_t c0 = t0; c0 < t1; c0 += CHUNK) {
    for (uint32_t k = lane; k < K; k += 64) mycnt[k] = 0;
    uint32_t key[ITEMS], rank[ITEMS];
    int64_t iss[ITEMS];
    int64_t carry_prev = 0;
    const int64_t wbase = c0 + (int64_t)w * 64 * ITEMS;
#pragma unroll
    for (int e = 0; e < ITEMS; e++) {
      const int64_t i = wbase + e * 64 + lane;
      const bool v = i < t1;
      int64_t x = v ? issue[i] : 0;
      uint64_t a = v ? addr[i] : 0;
      // previous request's issue time, for the order check
      int64_t prev = __shfl_up(x, 1);
      int64_t last_of_prev_item = carry_prev;
      carry_prev = __shfl(x, 63);
      if (lane == 0) prev = (e > 0) ? last_of_prev_item : ((i > 0 && v) ? issue[i - 1] : x);
      if (v) {
        if (x < 0 || x >= ISSUE_LIMIT) errb |= ERR_RANGE_TIME;
        if (i > 0 && x < prev) errb |= ERR_UNSORTED;
      }
      uint32_t k = v ? key_of<POW2>(g, lr, a) : KEY_NONE;
      if (v && k == KEY_NONE) complete[i] = x;  // native path: no modeled delay
      key[e] = k;
      iss[e] = x;
    }
    wave_rank(key, rank, mycnt, kbits);
    __syncthreads();
    cross_wave_offsets(wcnt, tot, K);
    __syncthreads();
#pragma unroll
    for (int e = 0; e < ITEMS; e++) {
      const uint32_t k = key[e];
      if (k != KEY_NONE) {
        const int64_t r0 = (int64_t)cnt[k] + mycnt[k] + rank[e];  // 0-based rank in tile
        atomicMax((long long *)&amax[k], (long long)(iss[e] - r0 * tR));
      }
    }
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < K; k += BLK) cnt[k] += tot[k];
    __syncthreads();
  }
  // tile aggregate per die queue: departure of the last request from an idle die
  const size_t row = (size_t)blockIdx.x * K;
  for (uint32_t k = threadIdx.x; k < K; k += BLK) {
    const uint32_t c = cnt[k];
    agg_cnt[row + k] = c;
    agg_A[row + k] = c ? (int64_t)c * tR + amax[k] : NEG;
  }
  if (errb) atomicOr(&ctl->err, errb);
}

// ------------------------------------------------------------------ k_tile_scan

// Per die queue, compose the tiles in order.  Block = 16 keys x 16 tile groups.
__global__ __launch_bounds__(BLK) void k_tile_scan(const uint32_t *__restrict__ agg_cnt,
                                                   const int64_t *__restrict__ agg_A, uint32_t nt,
                                                   uint32_t K, int64_t tR, const DevState *st,
                                                   int64_t *__restrict__ tin_L,
                                                   uint32_t *__restrict__ tin_base,
                                                   uint32_t *__restrict__ totals,
                                                   int64_t *__restrict__ dfnew, CallCtl *ctl) {
  __shared__ int64_t gA[16][16];
  __shared__ uint32_t gC[16][16];
  __shared__ int64_t inL[16][16];
  __shared__ uint32_t inB[16][16];
  if (agent_load32(&ctl->err)) return;
  const uint32_t kk = threadIdx.x & 15, tg = threadIdx.x >> 4;
  const uint32_t k = blockIdx.x * 16 + kk;
  const uint32_t per = (nt + 15) / 16;
  const uint32_t ta = tg * per, tb = min(nt, ta + per);
  // group aggregate: (A, count), A = NEG when empty
  int64_t A = NEG;
  uint32_t C = 0;
  if (k < K) {
    for (uint32_t t = ta; t < tb; t++) {
      const uint32_t c = agg_cnt[(size_t)t * K + k];
      if (c) {
        A = imax(agg_A[(size_t)t * K + k], A + (int64_t)c * tR);
        C += c;
      }
    }
  }
  gA[tg][kk] = A;
  gC[tg][kk] = C;
  __syncthreads();
  if (tg == 0 && k < K) {
    int64_t L = st->die_free[k];
    uint32_t base = 0;
    for (int q = 0; q < 16; q++) {
      inL[q][kk] = L;
      inB[q][kk] = base;
      if (gC[q][kk]) L = imax(gA[q][kk], L + (int64_t)gC[q][kk] * tR);
      base += gC[q][kk];
    }
    totals[k] = base;
    dfnew[k] = L;
    if (base) {
      atomicMax((long long *)&ctl->max_dd, (long long)L);
      if (L >= TIME_LIMIT) atomicOr(&ctl->err, ERR_OVERFLOW);
    }
  }
  __syncthreads();
  if (k < K) {
    int64_t L = inL[tg][kk];
    uint32_t base = inB[tg][kk];
    for (uint32_t t = ta; t < tb; t++) {
      tin_L[(size_t)t * K + k] = L;
      tin_base[(size_t)t * K + k] = base;
      const uint32_t c = agg_cnt[(size_t)t * K + k];
      if (c) L = imax(agg_A[(size_t)t * K + k], L + (int64_t)c * tR);
      base += c;
    }
  }
}

// ------------------------------------------------------------------ k_key_scan

// One block: die-queue segment starts, in-range count, time-cell grid.
__global__ __launch_bounds__(BLK) void k_key_scan(const uint32_t *__restrict__ totals, uint32_t K,
                                                  uint32_t *__restrict__ seg_start,
                                                  const int64_t *__restrict__ issue, uint32_t gmax,
                                                  uint32_t s0, CallCtl *ctl) {
  __shared__ uint32_t sh[WAVES];
  if (agent_load32(&ctl->err)) return;
  const uint32_t per = (K + BLK - 1) / BLK;
  const uint32_t a = threadIdx.x * per, b = min(K, a + per);
  uint32_t s = 0;
  for (uint32_t k = a; k < b; k++) s += totals[k];
  uint32_t ex;
  uint32_t tot = block_excl_sum(s, &ex, sh);
  for (uint32_t k = a; k < b; k++) {
    seg_start[k] = ex;
    ex += totals[k];
  }
  if (threadIdx.x == 0) {
    ctl->n_in = tot;
    if (tot == 0) {
      ctl->G = 0;
      ctl->shift = 0;
      ctl->cbase = 0;
    } else {
      const int64_t cbase = issue[0];
      const int64_t span = ctl->max_dd - cbase + 1;  // > 0: every die-done > issue[0]
      uint32_t sh2 = s0;
      while (sh2 < 62 && ((span - 1) >> sh2) + 1 > (int64_t)gmax) sh2++;
      ctl->cbase = cbase;
      ctl->shift = sh2;
      ctl->G = (uint32_t)(((span - 1) >> sh2) + 1);
    }
  }
}

// ------------------------------------------------------------------ k_die_scatter

// LDS: ranges | sval[CHUNK] i64 | L[K] i64 | cnt[K] u32 | gbase[K] u32 |
//      sloc[CHUNK] u16 | skey[CHUNK] u16 | wcnt[WAVES][K] u16 | tot[K] u16 | koff[K] u16
template <bool POW2>
__global__ __launch_bounds__(BLK) void k_die_scatter(
    const uint64_t *__restrict__ addr, const int64_t *__restrict__ issue, int64_t n, Geo g,
    RangeTable rt, int64_t tile_elems, const int64_t *__restrict__ tin_L,
    const uint32_t *__restrict__ tin_base, const uint32_t *__restrict__ seg_start,
    const uint32_t *__restrict__ totals, int64_t *__restrict__ DD, uint32_t *__restrict__ IX,
    uint32_t *__restrict__ LB, uint32_t gmax, CallCtl *ctl, uint32_t kbits) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ SegMax shseg[WAVES];
  __shared__ uint32_t shsum[WAVES];
  __shared__ uint32_t s_nvalid;
  if (agent_load32(&ctl->err)) return;
  LdsRanges *lr = (LdsRanges *)smem;
  const uint32_t K = g.K;
  int64_t *sval = (int64_t *)(smem + ((sizeof(LdsRanges) + 15) & ~size_t(15)));
  int64_t *L = sval + CHUNK;
  uint32_t *cnt = (uint32_t *)(L + K);
  uint32_t *gbase = cnt + K;
  uint16_t *sloc = (uint16_t *)(gbase + K);
  uint16_t *skey = sloc + CHUNK;
  uint16_t *wcnt = skey + CHUNK;
  uint16_t *tot = wcnt + WAVES * K;
  uint16_t *koff = tot + K;

  load_ranges(lr, rt);
  const size_t row = (size_t)blockIdx.x * K;
  for (uint32_t k = threadIdx.x; k < K; k += BLK) {
    cnt[k] = 0;
    L[k] = tin_L[row + k];
    gbase[k] = tin_base[row + k];  // die rank of the tile's first request of k
  }
  const int64_t cbase = ctl->cbase;
  const uint32_t shift = ctl->shift, G = ctl->G;
  __syncthreads();

  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * tile_elems;
  const int64_t t1 = imin(n, t0 + tile_elems);
  const int64_t tR = g.tR;
  uint16_t *mycnt = wcnt + w * K;
  const uint32_t Dk = g.Dk;

  for (int64_t c0 = t0; c0 < t1; c0 += CHUNK) {
    for (uint32_t k = lane; k < K; k += 64) mycnt[k] = 0;
    uint32_t key[ITEMS], rank[ITEMS];
    int64_t iss[ITEMS];
    const int64_t wbase = c0 + (int64_t)w * 64 * ITEMS;
#pragma unroll
    for (int e = 0; e < ITEMS; e++) {
      const int64_t i = wbase + e * 64 + lane;
      const bool v = i < t1;
      iss[e] = v ? issue[i] : 0;
      uint64_t a = v ? addr[i] : 0;
      key[e] = v ? key_of<POW2>(g, lr, a) : KEY_NONE;
    }
    wave_rank(key, rank, mycnt, kbits);
    __syncthreads();
    cross_wave_offsets(wcnt, tot, K);
    __syncthreads();
    // chunk offsets of each key's run: exclusive scan of tot over keys
    {
      const uint32_t per = (K + BLK - 1) / BLK;
      const uint32_t a = threadIdx.x * per, b = min(K, a + per);
      uint32_t s = 0;
      for (uint32_t k = a; k < b; k++) s += tot[k];
      uint32_t ex;
      uint32_t all = block_excl_sum(s, &ex, shsum);
      for (uint32_t k = a; k < b; k++) {
        koff[k] = (uint16_t)ex;
        ex += tot[k];
      }
      if (threadIdx.x == 0) s_nvalid = all;
    }
    __syncthreads();
    // stage in (key, rank) order
#pragma unroll
    for (int e = 0; e < ITEMS; e++) {
      const uint32_t k = key[e];
      if (k != KEY_NONE) {
        const uint32_t pos = koff[k] + mycnt[k] + rank[e];
        sval[pos] = iss[e];
        skey[pos] = (uint16_t)k;
        sloc[pos] = (uint16_t)(w * 64 * ITEMS + e * 64 + lane);
      }
    }
    __syncthreads();
    const uint32_t nv = s_nvalid;
    // segmented prefix max of v = issue - r0*tR over each key's run, then
    // die_done = (r0+1)*tR + max(M_k, prefix), M_k = L_k - cnt_k*tR
    {
      const uint32_t p0 = threadIdx.x * ITEMS;
      int64_t vals[ITEMS];
      SegMax agg = {0, NEG};
#pragma unroll
      for (int q = 0; q < ITEMS; q++) {
        const uint32_t p = p0 + q;
        if (p < nv) {
          const uint32_t k = skey[p];
          const uint32_t j = p - koff[k];
          const int64_t v = sval[p] - ((int64_t)cnt[k] + j) * tR;
          vals[q] = v;
          agg = seg_comb(agg, SegMax{j == 0, v});
        }
      }
      SegMax ex = block_excl_segmax(agg, shseg);
      int64_t run = ex.v;  // prefix of the segment continuing into this thread
#pragma unroll
      for (int q = 0; q < ITEMS; q++) {
        const uint32_t p = p0 + q;
        if (p < nv) {
          const uint32_t k = skey[p];
          const uint32_t j = p - koff[k];
          run = (j == 0) ? vals[q] : imax(run, vals[q]);
          const int64_t r0 = (int64_t)cnt[k] + j;
          const int64_t M = L[k] - (int64_t)cnt[k] * tR;
          sval[p] = (r0 + 1) * tR + imax(M, run);
        }
      }
    }
    __syncthreads();
    // write die-ordered (die_done, index); fill the cell table
    for (uint32_t p = threadIdx.x; p < nv; p += BLK) {
      const uint32_t k = skey[p];
      const uint32_t j = p - koff[k];
      const uint32_t r = gbase[k] + cnt[k] + j;  // die rank within this call
      const int64_t dd = sval[p];
      const size_t gpos = (size_t)seg_start[k] + r;
      DD[gpos] = dd;
      IX[gpos] = (uint32_t)(c0 + sloc[p]);
      const int64_t prev = (j > 0) ? sval[p - 1] : L[k];
      const int64_t cell = (dd - cbase) >> shift;
      const int64_t pcell = (r == 0) ? -1 : ((prev - cbase) >> shift);
      const uint32_t ch = k / Dk, dl = k - ch * Dk;
      uint32_t *lbrow = LB + (size_t)ch * (gmax + 1) * Dk + dl;
      for (int64_t c = pcell + 1; c <= cell; c++) lbrow[(size_t)c * Dk] = r;
      if (r + 1 == totals[k])
        for (int64_t c = cell + 1; c <= (int64_t)G; c++) lbrow[(size_t)c * Dk] = r + 1;
    }
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < K; k += BLK) {
      const uint32_t t = tot[k];
      if (t) {
        L[k] = sval[koff[k] + t - 1];
        cnt[k] += t;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ k_channel_merge

// (dd, idx) lexicographic order; idx is unique.
DEVI bool key_less(int64_t da, uint32_t ia, int64_t db, uint32_t ib) {
  return da < db || (da == db && ia < ib);
}

// Run containing position p: the last d with rb[d] <= p.
DEVI int run_of(const uint32_t *rb, int R, uint32_t p) {
  int lo = 0, hi = R;  // rb[0] <= p < rb[R]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (rb[mid] <= p) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Merge R sorted runs (boundaries rb[0..R], R a power of two) of m elements
// by pairwise merge levels in LDS.  Returns the buffer index holding the
// sorted result.
DEVI int lds_merge(int64_t *dd0, uint32_t *ix0, uint8_t *tg0, int64_t *dd1, uint32_t *ix1,
                   uint8_t *tg1, const uint32_t *rb, int R, uint32_t m, bool tags) {
  int cur = 0;
  for (int lvl = 0; (1 << lvl) < R; lvl++) {
    const int64_t *sd = cur ? dd1 : dd0;
    const uint32_t *si = cur ? ix1 : ix0;
    const uint8_t *st = cur ? tg1 : tg0;
    int64_t *dd = cur ? dd0 : dd1;
    uint32_t *di = cur ? ix0 : ix1;
    uint8_t *dt = cur ? tg0 : tg1;
    for (uint32_t p = threadIdx.x; p < m; p += BLK) {
      const int d = run_of(rb, R, p);
      const int gsel = d >> lvl;
      const uint32_t lo_g = rb[gsel << lvl];
      const int pg = gsel ^ 1;
      uint32_t lo = rb[pg << lvl], hi = rb[(pg + 1) << lvl];
      const int64_t x = sd[p];
      const uint32_t xi = si[p];
      // count partner elements less than x
      uint32_t a = lo, b = hi;
      while (a < b) {
        const uint32_t mid = (a + b) >> 1;
        if (key_less(sd[mid], si[mid], x, xi)) a = mid + 1;
        else b = mid;
      }
      const uint32_t out = rb[(gsel & ~1) << lvl] + (p - lo_g) + (a - lo);
      dd[out] = x;
      di[out] = xi;
      if (tags) dt[out] = st[p];
    }
    __syncthreads();
    cur ^= 1;
  }
  return cur;
}

struct MergeLds {
  int64_t dd[2][MCAP];
  uint32_t ix[2][MCAP];
  uint8_t tg[2][MCAP];
  uint32_t rb[MAX_RUNS + 1];
  uint32_t lo[MAX_RUNS];     // next global position to take, per run
  uint32_t hi[MAX_RUNS];     // end global position, per run
  uint32_t take[MAX_RUNS];
  uint32_t used[MAX_RUNS];
  int64_t shmax[WAVES];
  uint32_t shsum[WAVES];
  uint32_t ticket;
  uint32_t m;
  uint32_t safe;
  int64_t gin;
  int64_t qlast;
  uint32_t vstar_ok;
  int64_t vstar_d;
  uint32_t vstar_i;
};

// Sizes of cell j of channel c per run, from the cell table; returns total.
DEVI uint32_t cell_runs(MergeLds &S, const uint32_t *LB, const uint32_t *seg_start,
                        const uint32_t *totals, uint32_t c, uint32_t j, uint32_t Dk, uint32_t gmax,
                        int R) {
  if (threadIdx.x < (uint32_t)R) {
    const uint32_t d = threadIdx.x;
    uint32_t lo = 0, hi = 0;
    if (d < Dk) {
      const uint32_t k = c * Dk + d;
      if (totals[k]) {
        const uint32_t *lbrow = LB + (size_t)c * (gmax + 1) * Dk + d;
        lo = lbrow[(size_t)j * Dk];
        hi = lbrow[(size_t)(j + 1) * Dk];
      }
      lo += seg_start[k];
      hi += seg_start[k];
    }
    S.lo[d] = lo;
    S.hi[d] = hi;
  }
  __syncthreads();
  uint32_t tot = 0;
  if (threadIdx.x == 0) {
    for (int d = 0; d < R; d++) tot += S.hi[d] - S.lo[d];
    S.m = tot;
  }
  __syncthreads();
  return S.m;
}

// Decoupled look-back (wave 0): channel clock entering cell j of channel c.
DEVI int64_t look_back(const uint64_t *st_agg, const uint64_t *st_incl, const uint32_t *LB,
                       const uint32_t *totals, const DevState *st, uint32_t c, uint32_t j,
                       uint32_t Dk, uint32_t gmax, int64_t xfer) {
  int64_t A = NEG, B = 0;  // composition of the cells between jj and j (identity)
  const uint32_t lane = lane_id();
  int64_t jj = (int64_t)j - 1;
  while (true) {
    if (jj < 0) {
      const int64_t f0 = st->chan_free[c];
      return imax(A, f0 + B);
    }
    const size_t sidx = (size_t)c * gmax + jj;
    const uint64_t wi = agent_load(&st_incl[sidx]);
    if (wi) return imax(A, dec_time(wi) + B);
    const uint64_t wa = agent_load(&st_agg[sidx]);
    if (wa) {
      // size of cell jj from the cell table (lanes over dies)
      uint32_t sz = 0;
      if (lane < Dk) {
        const uint32_t k = c * Dk + lane;
        if (totals[k]) {
          const uint32_t *lbrow = LB + (size_t)c * (gmax + 1) * Dk + lane;
          sz = lbrow[(size_t)(jj + 1) * Dk] - lbrow[(size_t)jj * Dk];
        }
      }
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) sz += __shfl_xor(sz, d);
      const int64_t Bj = (int64_t)sz * xfer;
      A = imax(A, dec_time(wa) + B);
      B += Bj;
      jj--;
      continue;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Load runs [lo[d], lo[d]+take[d]) into buffer 0; rb gets the boundaries.
DEVI uint32_t load_runs(MergeLds &S, const int64_t *DD, const uint32_t *IX, int R, bool tags) {
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int d = 0; d < R; d++) {
      S.rb[d] = s;
      s += S.take[d];
    }
    S.rb[R] = s;
  }
  __syncthreads();
  const uint32_t m = S.rb[R];
  for (uint32_t p = threadIdx.x; p < m; p += BLK) {
    const int d = run_of(S.rb, R, p);
    const uint32_t src = S.lo[d] + (p - S.rb[d]);
    S.dd[0][p] = DD[src];
    S.ix[0][p] = IX[src];
    if (tags) S.tg[0][p] = (uint8_t)d;
  }
  __syncthreads();
  return m;
}

// Prefix max of v_p = dd_p - p*xfer over buffer `b`, in place, for p < m.
// Returns nothing; S.qlast receives the value at m-1.
DEVI void prefix_q(MergeLds &S, int b, uint32_t m, int64_t xfer) {
  constexpr int E = MCAP / BLK;
  const uint32_t p0 = threadIdx.x * E;
  int64_t loc = NEG;
#pragma unroll
  for (int q = 0; q < E; q++) {
    const uint32_t p = p0 + q;
    if (p < m) loc = imax(loc, S.dd[b][p] - (int64_t)p * xfer);
  }
  int64_t run = block_excl_max(loc, S.shmax);
#pragma unroll
  for (int q = 0; q < E; q++) {
    const uint32_t p = p0 + q;
    if (p < m) {
      run = imax(run, S.dd[b][p] - (int64_t)p * xfer);
      S.dd[b][p] = run;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) S.qlast = m ? S.dd[b][m - 1] : NEG;
  __syncthreads();
}

// One pass over an oversized cell in bounded rounds.  Each round loads at
// most MCAP/R requests per run, merges them, and serves the prefix that no
// unloaded request can precede.  Returns the channel clock after the cell;
// writes complete[] when `emit`.
DEVI int64_t stream_cell(MergeLds &S, const int64_t *DD, const uint32_t *IX, int R, int64_t gstart,
                         int64_t xfer, bool emit, int64_t *complete, uint32_t *errb,
                         const uint32_t *lo0, const uint32_t *hi0) {
  if (threadIdx.x < (uint32_t)R) {
    S.lo[threadIdx.x] = lo0[threadIdx.x];
    S.hi[threadIdx.x] = hi0[threadIdx.x];
  }
  __syncthreads();
  int64_t G = gstart;
  const uint32_t quota = MCAP / R;
  while (true) {
    if (threadIdx.x == 0) {
      uint32_t rem = 0;
      for (int d = 0; d < R; d++) rem += S.hi[d] - S.lo[d];
      const bool all = rem <= MCAP;
      S.vstar_ok = 0;
      for (int d = 0; d < R; d++) {
        const uint32_t r = S.hi[d] - S.lo[d];
        S.take[d] = all ? r : min(r, quota);
        S.used[d] = 0;
      }
      S.m = rem;
    }
    __syncthreads();
    if (S.m == 0) break;
    const uint32_t m = load_runs(S, DD, IX, R, true);
    // bound: smallest last-loaded key among runs with requests left behind
    if (threadIdx.x == 0) {
      bool ok = false;
      int64_t vd = 0;
      uint32_t vi = 0;
      for (int d = 0; d < R; d++) {
        if (S.take[d] < S.hi[d] - S.lo[d] && S.take[d] > 0) {
          const uint32_t q = S.rb[d + 1] - 1;
          if (!ok || key_less(S.dd[0][q], S.ix[0][q], vd, vi)) {
            vd = S.dd[0][q];
            vi = S.ix[0][q];
            ok = true;
          }
        }
      }
      S.vstar_ok = ok;
      S.vstar_d = vd;
      S.vstar_i = vi;
    }
    __syncthreads();
    const int b = lds_merge(S.dd[0], S.ix[0], S.tg[0], S.dd[1], S.ix[1], S.tg[1], S.rb, R, m, true);
    // safe prefix: elements <= vstar
    if (threadIdx.x == 0) {
      uint32_t safe = m;
      if (S.vstar_ok) {
        uint32_t a = 0, c = m;
        while (a < c) {
          const uint32_t mid = (a + c) >> 1;
          if (!key_less(S.vstar_d, S.vstar_i, S.dd[b][mid], S.ix[b][mid])) a = mid + 1;
          else c = mid;
        }
        safe = a;
      }
      S.safe = safe;
    }
    __syncthreads();
    const uint32_t safe = S.safe;
    for (uint32_t p = threadIdx.x; p < safe; p += BLK) atomicAdd(&S.used[S.tg[b][p]], 1u);
    prefix_q(S, b, safe, xfer);
    if (emit) {
      for (uint32_t p = threadIdx.x; p < safe; p += BLK) {
        const int64_t cpl = (int64_t)(p + 1) * xfer + imax(G, S.dd[b][p]);
        if (cpl >= TIME_LIMIT) *errb |= ERR_OVERFLOW;
        complete[S.ix[b][p]] = cpl;
      }
    }
    G = (int64_t)safe * xfer + imax(G, S.qlast);
    __syncthreads();
    if (threadIdx.x < (uint32_t)R) S.lo[threadIdx.x] += S.used[threadIdx.x];
    __syncthreads();
  }
  return G;
}

__global__ __launch_bounds__(BLK) void k_channel_merge(
    const int64_t *__restrict__ DD, const uint32_t *__restrict__ IX, const uint32_t *__restrict__ LB,
    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ totals, Geo g,
    CallCtl *ctl, uint64_t *st_agg, uint64_t *st_incl, const DevState *st,
    int64_t *__restrict__ cfnew, int64_t *__restrict__ complete, uint32_t gmax) {
  extern __shared__ __align__(16) unsigned char smem[];
  MergeLds &S = *(MergeLds *)smem;
  if (agent_load32(&ctl->err)) return;
  const uint32_t G = ctl->G, C = g.C, Dk = g.Dk;
  const uint64_t ncell = (uint64_t)G * C;
  int R = 1;
  while (R < (int)Dk) R <<= 1;
  const int64_t xfer = g.xfer;
  uint32_t errb = 0;
  uint32_t lo0[1], hi0[1];
  (void)lo0;
  (void)hi0;
  __shared__ uint32_t slo[MAX_RUNS], shi[MAX_RUNS];
  while (true) {
    if (threadIdx.x == 0) S.ticket = atomicAdd(&ctl->ticket, 1u);
    __syncthreads();
    const uint32_t tk = S.ticket;
    __syncthreads();
    if ((uint64_t)tk >= ncell) break;
    const uint32_t c = tk % C, j = tk / C;
    const uint32_t m = cell_runs(S, LB, seg_start, totals, c, j, Dk, gmax, R);
    const size_t sidx = (size_t)c * gmax + j;
    int64_t A;
    bool resident = m <= MCAP;
    int b = 0;
    if (resident) {
      if (threadIdx.x < (uint32_t)R) S.take[threadIdx.x] = S.hi[threadIdx.x] - S.lo[threadIdx.x];
      __syncthreads();
      load_runs(S, DD, IX, R, false);
      b = lds_merge(S.dd[0], S.ix[0], S.tg[0], S.dd[1], S.ix[1], S.tg[1], S.rb, R, m, false);
      prefix_q(S, b, m, xfer);
      A = m ? (int64_t)m * xfer + S.qlast : NEG;
    } else {
      if (threadIdx.x < (uint32_t)R) {
        slo[threadIdx.x] = S.lo[threadIdx.x];
        shi[threadIdx.x] = S.hi[threadIdx.x];
      }
      __syncthreads();
      A = stream_cell(S, DD, IX, R, NEG, xfer, false, complete, &errb, slo, shi);
    }
    // publish the cell aggregate, then find the incoming channel clock
    if (threadIdx.x == 0) agent_store(&st_agg[sidx], enc_time(A));
    if (threadIdx.x < 64) {
      const int64_t gin = look_back(st_agg, st_incl, LB, totals, st, c, j, Dk, gmax, xfer);
      if (threadIdx.x == 0) {
        S.gin = gin;
        const int64_t gout = imax(A, gin + (int64_t)m * xfer);
        agent_store(&st_incl[sidx], enc_time(gout));
        if (j + 1 == G) cfnew[c] = gout;
      }
    }
    __syncthreads();
    const int64_t gin = S.gin;
    if (resident) {
      for (uint32_t p = threadIdx.x; p < m; p += BLK) {
        const int64_t cpl = (int64_t)(p + 1) * xfer + imax(gin, S.dd[b][p]);
        if (cpl >= TIME_LIMIT) errb |= ERR_OVERFLOW;
        complete[S.ix[b][p]] = cpl;
      }
    } else {
      stream_cell(S, DD, IX, R, gin, xfer, true, complete, &errb, slo, shi);
    }
    __syncthreads();
  }
  if (errb) atomicOr(&ctl->err, errb);
}

// ------------------------------------------------------------------ k_finalize

__global__ __launch_bounds__(BLK) void k_finalize(int64_t *__restrict__ complete, int64_t n,
                                                  CallCtl *ctl, DevState *st,
                                                  const int64_t *__restrict__ dfnew,
                                                  const uint32_t *__restrict__ totals,
                                                  const int64_t *__restrict__ cfnew, uint32_t K,
                                                  uint32_t C) {
  const uint32_t err = agent_load32(&ctl->err);
  if (err) {
    for (int64_t i = (int64_t)blockIdx.x * BLK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLK)
      complete[i] = HBF_TIME_ERROR;
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&st->sticky, err);
    return;
  }
  if (blockIdx.x != 0) return;
  for (uint32_t k = threadIdx.x; k < K; k += BLK)
    if (totals[k]) st->die_free[k] = dfnew[k];
  if (ctl->G)
    for (uint32_t c = threadIdx.x; c < C; c += BLK) st->chan_free[c] = cfnew[c];
}

// ------------------------------------------------------------------ classify + reset

template <bool POW2>
__global__ __launch_bounds__(BLK) void k_classify(const uint64_t *__restrict__ addr, int64_t n,
                                                  uint64_t *__restrict__ map, Geo g, RangeTable rt,
                                                  DevState *st) {
  __shared__ LdsRanges lr;
  load_ranges(&lr, rt);
  __syncthreads();
  uint32_t errb = 0;
  for (int64_t i = (int64_t)blockIdx.x * BLK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLK) {
    const uint64_t a = addr[i];
    const int r = find_range(&lr, a);
    uint64_t word = 0;
    if (r >= 0) {
      const Loc L = map_page<POW2>(g, dev_page<POW2>(g, &lr, r, a));
      if (L.page > 0xffffffffull) {
        errb |= ERR_MAP;
      } else {
        word = (uint64_t(1) << 63) | ((uint64_t)lr.rid[r] << 56) | ((uint64_t)L.plane << 50) |
               ((uint64_t)L.die << 42) | ((uint64_t)L.ch << 32) | L.page;
      }
    }
    map[i] = word;
  }
  if (errb) atomicOr(&st->sticky, errb);
}

__global__ void k_reset(DevState *st) {
  for (uint32_t k = threadIdx.x; k < MAX_KEYS; k += blockDim.x) st->die_free[k] = NEG;
  for (uint32_t c = threadIdx.x; c < MAX_CHANNELS; c += blockDim.x) st->chan_free[c] = NEG;
}

// ------------------------------------------------------------------ launchers

const char *const kKernelNames[] = {"k_prologue",    "k_die_reduce",    "k_tile_scan", "k_key_scan",
                                    "k_die_scatter", "k_channel_merge", "k_finalize"};
const int kNumTimedKernels = 7;

static uint32_t bits_for(uint32_t K) {
  uint32_t b = 0;
  while ((1u << b) < K) b++;
  return b ? b : 1;
}

static size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

size_t lds_die_reduce(uint32_t K) {
  return align16(sizeof(LdsRanges)) + K * (8 + 4) + WAVES * K * 2 + K * 2;
}
size_t lds_die_scatter(uint32_t K) {
  return align16(sizeof(LdsRanges)) + CHUNK * 8 + K * (8 + 4 + 4) + CHUNK * 4 + WAVES * K * 2 + K * 4;
}

hipError_t launch_time_requests(const Geo &g, const RangeTable &rt, const Layout &Lo, char *ws,
                                DevState *st, const uint64_t *addr, const int64_t *issue,
                                int64_t *complete, hipStream_t s, hipEvent_t *ev, int n_ev) {
  CallCtl *ctl = (CallCtl *)(ws + Lo.off_ctl);
  uint32_t *agg_cnt = (uint32_t *)(ws + Lo.off_agg_cnt);
  int64_t *agg_A = (int64_t *)(ws + Lo.off_agg_A);
  int64_t *tin_L = (int64_t *)(ws + Lo.off_tin_L);
  uint32_t *tin_base = (uint32_t *)(ws + Lo.off_tin_base);
  uint32_t *totals = (uint32_t *)(ws + Lo.off_totals);
  uint32_t *seg = (uint32_t *)(ws + Lo.off_seg);
  int64_t *dfnew = (int64_t *)(ws + Lo.off_dfnew);
  int64_t *cfnew = (int64_t *)(ws + Lo.off_cfnew);
  int64_t *DD = (int64_t *)(ws + Lo.off_dd);
  uint32_t *IX = (uint32_t *)(ws + Lo.off_ix);
  uint32_t *LB = (uint32_t *)(ws + Lo.off_lb);
  uint64_t *st_agg = (uint64_t *)(ws + Lo.off_st_agg);
  uint64_t *st_incl = (uint64_t *)(ws + Lo.off_st_incl);
  const uint32_t kbits = bits_for(g.K);
  const bool p2 = g.pow2 != 0;
  const size_t nst = (size_t)g.C * Lo.gmax;
  int evi = 0;
  auto mark = [&]() {
    if (ev && evi < n_ev) hipEventRecord(ev[evi++], s);
  };
  hipError_t e;
  mark();
  {
    size_t blocks = (nst + BLK - 1) / BLK;
    if (blocks > 2048) blocks = 2048;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_prologue, dim3((uint32_t)blocks), dim3(BLK), 0, s, ctl, st_agg, st_incl, nst);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  {
    const size_t lds = lds_die_reduce(g.K);
    if (p2)
      hipLaunchKernelGGL(k_die_reduce<true>, dim3(Lo.nt), dim3(BLK), lds, s, addr, issue, Lo.n, complete,
                         g, rt, Lo.tile_elems, agg_cnt, agg_A, ctl, kbits);
    else
      hipLaunchKernelGGL(k_die_reduce<false>, dim3(Lo.nt), dim3(BLK), lds, s, addr, issue, Lo.n,
                         complete, g, rt, Lo.tile_elems, agg_cnt, agg_A, ctl, kbits);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  hipLaunchKernelGGL(k_tile_scan, dim3((g.K + 15) / 16), dim3(BLK), 0, s, agg_cnt, agg_A, Lo.nt, g.K,
                     g.tR, st, tin_L, tin_base, totals, dfnew, ctl);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  hipLaunchKernelGGL(k_key_scan, dim3(1), dim3(BLK), 0, s, totals, g.K, seg, issue, Lo.gmax, Lo.s0, ctl);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  {
    const size_t lds = lds_die_scatter(g.K);
    if (p2)
      hipLaunchKernelGGL(k_die_scatter<true>, dim3(Lo.nt), dim3(BLK), lds, s, addr, issue, Lo.n, g, rt,
                         Lo.tile_elems, tin_L, tin_base, seg, totals, DD, IX, LB, Lo.gmax, ctl, kbits);
    else
      hipLaunchKernelGGL(k_die_scatter<false>, dim3(Lo.nt), dim3(BLK), lds, s, addr, issue, Lo.n, g, rt,
                         Lo.tile_elems, tin_L, tin_base, seg, totals, DD, IX, LB, Lo.gmax, ctl, kbits);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  {
    int dev = 0, ncu = 256;
    hipGetDevice(&dev);
    hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    const uint32_t blocks = (uint32_t)ncu * 2;
    hipLaunchKernelGGL(k_channel_merge, dim3(blocks), dim3(BLK), sizeof(MergeLds), s, DD, IX, LB, seg,
                       totals, g, ctl, st_agg, st_incl, st, cfnew, complete, Lo.gmax);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  {
    int64_t blocks = (Lo.n + BLK - 1) / BLK;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_finalize, dim3((uint32_t)blocks), dim3(BLK), 0, s, complete, Lo.n, ctl, st, dfnew,
                       totals, cfnew, g.K, g.C);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  return hipSuccess;
}

hipError_t launch_classify(const Geo &g, const RangeTable &rt, DevState *st, const uint64_t *addr,
                           int64_t n, uint64_t *map, hipStream_t s) {
  int64_t blocks = (n + BLK - 1) / BLK;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  if (g.pow2)
    hipLaunchKernelGGL(k_classify<true>, dim3((uint32_t)blocks), dim3(BLK), 0, s, addr, n, map, g, rt, st);
  else
    hipLaunchKernelGGL(k_classify<false>, dim3((uint32_t)blocks), dim3(BLK), 0, s, addr, n, map, g, rt, st);
  return hipGetLastError();
}

hipError_t launch_reset(DevState *st, hipStream_t s) {
  hipLaunchKernelGGL(k_reset, dim3(1), dim3(BLK), 0, s, st);
  return hipGetLastError();
}

hipError_t set_lds_limits(uint32_t K) {
  hipError_t e;
  const int a = (int)lds_die_reduce(K), b = (int)lds_die_scatter(K), c = (int)sizeof(MergeLds);
  if ((e = hipFuncSetAttribute((const void *)k_die_reduce<true>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, a)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void *)k_die_reduce<false>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, a)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void *)k_die_scatter<true>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, b)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void *)k_die_scatter<false>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, b)) != hipSuccess)
    return e;
  return hipFuncSetAttribute((const void *)k_channel_merge, hipFuncAttributeMaxDynamicSharedMemorySize,
                             c);
}

}  // namespace hbf
