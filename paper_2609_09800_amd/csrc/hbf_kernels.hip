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
//   k_cell_chan    per (time window, channel group), in window order: merge
//                  each cell's die runs by (die-done, index), publish the
//                  cell's channel term, take the term entering it by a
//                  decoupled look-back over earlier windows, and write
//                  complete[] in request order (staged by index in LDS
//                  where the window's requests cluster).
//   k_cell_agg, k_cell_scan, k_cell_rest
//                  the same stage as reduce, scan and reduce again, for
//                  grids whose cells are too wide for the bucket merge.
//   k_finalize     fail-closed error fill, or commit of the new clocks.
//
// A die emits at most one request per t_read_ns, so a time cell of width
// 2^shift <= T * t_read_ns holds at most T requests per die, and a bucket
// of width 2^floor(log2 t_read_ns) at most one: cells are bounded by
// construction and merge without searching.
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdint.h>

#include "hbf_device.h"
#include "hbf_internal.h"

namespace hbf {

// ------------------------------------------------------------------ k_prologue

__global__ void k_prologue(CallCtl *ctl) {
  if (threadIdx.x == 0) {
    ctl->err = 0;
    ctl->n_in = 0;
    ctl->G = 0;
    ctl->shift = 0;
    ctl->max_dd = NEG;
    ctl->max_cpl = NEG;
    ctl->cbase = 0;
    ctl->n_rest = 0;
    ctl->wctr = 0;
  }
}

// ------------------------------------------------------------------ k_die_reduce


// Die time of the first g admissions of a die queue in one call when the
// first R of them each also carry a refresh quantum (Section D4): the sum of
// their services, g*tR + min(g, R)*tQ.  With R = 0 it is the plain g*tR.
DEVI int64_t svc_sum(uint32_t g, uint32_t R, int64_t tR, int64_t tQ) {
  return (int64_t)g * tR + (int64_t)min(g, R) * tQ;
}

// With refresh quanta pending (REF) the service of a die queue's request
// depends on its rank in the call, so the tile aggregate is kept in global
// form, max over the tile of issue - svc_sum(global rank), with the global
// ranks of the tile's first requests taken from a count pass (tin_base).
// LDS: ranges | amax[K] i64 | cmax[K] i64 | cnt[K] u32 | wcnt[DWAVES][K] u16 | tot[K] u16 | refp[K] u32 |
//      tag[DWAVES][K] u32
template <bool POW2, bool REF>
__global__ __launch_bounds__(DBLK) void k_die_reduce(const uint64_t *__restrict__ addr,
                                                    const int64_t *__restrict__ issue, int64_t n,
                                                    int64_t *__restrict__ complete, Geo g,
                                                    RangeTable rt, int64_t tile_elems,
                                                    uint32_t *__restrict__ agg_cnt,
                                                    int64_t *__restrict__ agg_A,
                                                    uint32_t *__restrict__ KR, CallCtl *ctl,
                                                    const uint32_t *__restrict__ tin_base,
                                                    const DevState *st) {
  extern __shared__ __align__(16) unsigned char smem[];
  LdsRanges *lr = (LdsRanges *)smem;
  const uint32_t K = g.K;
  int64_t *amax = (int64_t *)(smem + ((sizeof(LdsRanges) + 15) & ~size_t(15)));
  int64_t *cmax = amax + K;  // this chunk's max of issue - (rank in chunk)*tR, per key
  uint32_t *cnt = (uint32_t *)(cmax + K);
  uint16_t *wcnt = (uint16_t *)(cnt + K);
  uint16_t *tot = wcnt + DWAVES * K;
  // REF: pending quanta per key, read once per block (4-byte aligned: K may be odd)
  uint32_t *refp = (uint32_t *)(((uintptr_t)(tot + K) + 3) & ~(uintptr_t)3);
  uint32_t *tags = refp + K;

  // per-queue LDS state is indexed by the queue's LDS slot (lslot); global
  // per-queue arrays by the queue itself
  load_ranges(lr, rt);
  for (uint32_t li = threadIdx.x; li < K; li += DBLK) {
    const uint32_t k = lkey(g, li);
    // REF: cnt holds the call-wide rank of the tile's next request of k
    cnt[li] = REF ? tin_base[(size_t)blockIdx.x * K + k] : 0;
    amax[li] = NEG;
    cmax[li] = NEG;
    if (REF) refp[li] = st->ref_pend[k];
  }
  __syncthreads();
  const RangeReg rr = range_reg(lr);

  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * tile_elems;
  const int64_t t1 = imin(n, t0 + tile_elems);
  const int64_t tR = g.tR;
  uint32_t errb = 0;
  uint16_t *mycnt = wcnt + w * K;

  // the next chunk's requests are loaded while this one is ranked
  int64_t nx[DITEMS], nb = 0;
  uint64_t na[DITEMS];
  auto fetch = [&](int64_t cc) {
    const int64_t wb = cc + (int64_t)w * 64 * DITEMS;
#pragma unroll
    for (int e = 0; e < DITEMS; e++) {
      const int64_t i = wb + e * 64 + lane;
      const bool v = i < t1;
      nx[e] = v ? issue[i] : 0;
      na[e] = v ? addr[i] : 0;
    }
    nb = (lane == 0 && wb > 0 && wb < t1) ? issue[wb - 1] : 0;
  };
  if (t0 < t1) fetch(t0);
  for (int64_t c0 = t0; c0 < t1; c0 += CHUNK) {
    for (uint32_t k = lane; k < K; k += 64) mycnt[k] = 0;
    uint32_t key[DITEMS], rank[DITEMS];
    int64_t iss[DITEMS];
    int64_t cx[DITEMS];
    uint64_t ca[DITEMS];
#pragma unroll
    for (int e = 0; e < DITEMS; e++) {
      cx[e] = nx[e];
      ca[e] = na[e];
    }
    const int64_t before = nb;  // issue time preceding this wave's first request
    if (c0 + CHUNK < t1) fetch(c0 + CHUNK);
    int64_t carry_prev = 0;
    const int64_t wbase = c0 + (int64_t)w * 64 * DITEMS;
#pragma unroll
    for (int e = 0; e < DITEMS; e++) {
      const int64_t i = wbase + e * 64 + lane;
      const bool v = i < t1;
      const int64_t x = cx[e];
      const uint64_t a = ca[e];
      // previous request's issue time, for the order check
      int64_t prev = dpp64<DPP_WAVE_SHR1, 0xF>(x, x);  // lane l - 1's issue time
      int64_t last_of_prev_item = carry_prev;
      carry_prev = lane63(x);
      if (lane == 0) prev = (e > 0) ? last_of_prev_item : ((i > 0 && v) ? before : x);
      if (v) {
        if (x < 0 || x >= ISSUE_LIMIT) errb |= ERR_RANGE_TIME;
        if (i > 0 && x < prev) errb |= ERR_UNSORTED;
      }
      uint32_t k = v ? key_of<POW2>(g, lr, rr, a) : KEY_NONE;
      if (v && k == KEY_NONE) complete[i] = x;  // native path: no modeled delay
      key[e] = k == KEY_NONE ? KEY_NONE : lslot(g, k);
      iss[e] = x;
    }
    wave_rank(key, rank, mycnt, tags + w * K);
    __syncthreads();
    cross_wave_offsets(wcnt, tot, K);
    __syncthreads();
#pragma unroll
    for (int e = 0; e < DITEMS; e++) {
      const uint32_t k = key[e];
      const int64_t i = wbase + e * 64 + lane;
      if (k != KEY_NONE) {
        const uint32_t rc = mycnt[k] + rank[e];  // rank among key k in the chunk
        if (REF)
          atomicMax((long long *)&amax[k],
                    (long long)(iss[e] - svc_sum(cnt[k] + rc, refp[k], tR, g.tQ)));
        else
          atomicMax((long long *)&cmax[k], (long long)(iss[e] - (int64_t)mul32(rc, (uint32_t)tR)));
        KR[i] = (k << 16) | rc;
      } else if (i < t1) {
        KR[i] = (uint32_t)KEY_NONE << 16;
      }
    }
    __syncthreads();
    // fold the chunk into the tile: ranks in the tile are cnt[k] + rank in chunk
    for (uint32_t k = threadIdx.x; k < K; k += DBLK) {
      const uint32_t t = tot[k];
      if (t) {
        if (!REF) {
          amax[k] = imax(amax[k], cmax[k] - (int64_t)mul32(cnt[k], (uint32_t)tR));
          cmax[k] = NEG;
        }
        cnt[k] += t;
      }
    }
    __syncthreads();
  }
  const size_t row = (size_t)blockIdx.x * K;
  for (uint32_t li = threadIdx.x; li < K; li += DBLK) {
    const uint32_t k = lkey(g, li);
    if (REF) {  // global form; the counts came from the count pass
      agg_A[row + k] = amax[li];
    } else {    // departure of the tile's last request of k from an idle die
      const uint32_t c = cnt[li];
      agg_cnt[row + k] = c;
      agg_A[row + k] = c ? (int64_t)c * tR + amax[li] : NEG;
    }
  }
  if (errb) atomicOr(&ctl->err, errb);
}

// Count pass of the refresh path: per tile, the in-range requests of each
// die queue (no ranks, no times).
template <bool POW2>
__global__ __launch_bounds__(DBLK) void k_die_count(const uint64_t *__restrict__ addr, int64_t n, Geo g,
                                                   RangeTable rt, int64_t tile_elems,
                                                   uint32_t *__restrict__ agg_cnt) {
  extern __shared__ __align__(16) unsigned char smem[];
  LdsRanges *lr = (LdsRanges *)smem;
  uint32_t *cnt = (uint32_t *)(smem + ((sizeof(LdsRanges) + 15) & ~size_t(15)));
  const uint32_t K = g.K;
  load_ranges(lr, rt);
  for (uint32_t k = threadIdx.x; k < K; k += DBLK) cnt[k] = 0;
  __syncthreads();
  const int64_t t0 = (int64_t)blockIdx.x * tile_elems;
  const int64_t t1 = imin(n, t0 + tile_elems);
  const RangeReg rr = range_reg(lr);
  for (int64_t i = t0 + threadIdx.x; i < t1; i += DBLK) {
    const uint32_t k = key_of<POW2>(g, lr, rr, addr[i]);
    if (k != KEY_NONE) atomicAdd(&cnt[lslot(g, k)], 1u);
  }
  __syncthreads();
  for (uint32_t li = threadIdx.x; li < K; li += DBLK) agg_cnt[(size_t)blockIdx.x * K + lkey(g, li)] = cnt[li];
}

// Refresh path: per die queue, the call-wide rank of each tile's first
// request (exclusive prefix over tiles) and the queue's total.  One wave
// per die queue, lane = contiguous group of tiles.
__global__ __launch_bounds__(BLK) void k_tile_count(const uint32_t *__restrict__ agg_cnt, uint32_t nt, uint32_t K,
                                                    uint32_t *__restrict__ tin_base,
                                                    uint32_t *__restrict__ totals) {
  const uint32_t lane = lane_id();
  const uint32_t k = blockIdx.x * WAVES + (threadIdx.x >> 6);
  if (k >= K) return;  // whole wave
  const uint32_t per = (nt + 63) / 64;
  const uint32_t ta = min(nt, lane * per), tb = min(nt, ta + per);
  uint32_t C = 0;
  for (uint32_t t = ta; t < tb; t++) C += agg_cnt[(size_t)t * K + k];
  uint32_t base = wave_excl_sum(C);
  if (lane == 63) totals[k] = base + C;
  for (uint32_t t = ta; t < tb; t++) {
    tin_base[(size_t)t * K + k] = base;
    base += agg_cnt[(size_t)t * K + k];
  }
}

// Refresh path: per die queue, the clock entering each tile from the
// global-form tile maxima M_t:  L = svc_sum(base) + max(f0, max of M before).
__global__ __launch_bounds__(BLK) void k_tile_scan_ref(const int64_t *__restrict__ agg_A, uint32_t nt, Geo g,
                                                       const DevState *st, const uint32_t *__restrict__ tin_base,
                                                       const uint32_t *__restrict__ totals,
                                                       int64_t *__restrict__ tin_L,
                                                       int64_t *__restrict__ dfnew, CallCtl *ctl) {
  if (agent_load32(&ctl->err)) return;
  const uint32_t lane = lane_id(), K = g.K;
  const uint32_t k = blockIdx.x * WAVES + (threadIdx.x >> 6);
  if (k >= K) return;  // whole wave
  const uint32_t per = (nt + 63) / 64;
  const uint32_t ta = min(nt, lane * per), tb = min(nt, ta + per);
  int64_t M = NEG;
  for (uint32_t t = ta; t < tb; t++) M = imax(M, agg_A[(size_t)t * K + k]);
  const int64_t inc = wave_incl_max(M);
  int64_t run = __shfl_up(inc, 1);
  if (lane == 0) run = NEG;
  const int64_t f0 = st->die_free[k];
  const uint32_t R = st->ref_pend[k];
  if (lane == 63) {
    const uint32_t tot = totals[k];
    if (tot) {
      const int64_t Lend = svc_sum(tot, R, g.tR, g.tQ) + imax(f0, inc);
      dfnew[k] = Lend;
      atomicMax((long long *)&ctl->max_dd, (long long)Lend);
      if (Lend >= TIME_LIMIT) atomicOr(&ctl->err, ERR_OVERFLOW);
    }
  }
  for (uint32_t t = ta; t < tb; t++) {
    tin_L[(size_t)t * K + k] = svc_sum(tin_base[(size_t)t * K + k], R, g.tR, g.tQ) + imax(f0, run);
    run = imax(run, agg_A[(size_t)t * K + k]);
  }
}

// Per die queue, compose the tiles in order.  One wave per die queue, lane g
// holding a contiguous group of tiles: each lane folds its group, a wave
// scan composes the groups, and each lane walks its group again writing the
// clock and rank entering every tile.  Composition of (A, count) segments in
// order: (A1, c1) then (A2, c2) = (max(A2, A1 + c2*tR), c1 + c2), A = NEG
// when empty; a clock L entering a segment leaves as max(A, L + c*tR).
__global__ __launch_bounds__(BLK) void k_tile_scan(const uint32_t *__restrict__ agg_cnt,
                                                   const int64_t *__restrict__ agg_A, uint32_t nt,
                                                   uint32_t K, int64_t tR, const DevState *st,
                                                   int64_t *__restrict__ tin_L,
                                                   uint32_t *__restrict__ tin_base,
                                                   uint32_t *__restrict__ totals,
                                                   int64_t *__restrict__ dfnew, CallCtl *ctl) {
  if (agent_load32(&ctl->err)) return;
  const uint32_t lane = lane_id();
  const uint32_t k = blockIdx.x * WAVES + (threadIdx.x >> 6);
  if (k >= K) return;  // whole wave
  const uint32_t per = (nt + 63) / 64;
  const uint32_t ta = min(nt, lane * per), tb = min(nt, ta + per);
  int64_t A = NEG;
  uint32_t C = 0;
  for (uint32_t t = ta; t < tb; t++) {
    const uint32_t c = agg_cnt[(size_t)t * K + k];
    if (c) {
      A = imax(agg_A[(size_t)t * K + k], A + (int64_t)c * tR);
      C += c;
    }
  }
  // inclusive scan over the lanes' groups
  int64_t iA = A;
  uint32_t iC = C;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t pA = __shfl_up(iA, d);
    const uint32_t pC = __shfl_up(iC, d);
    if (lane >= (uint32_t)d) {
      iA = imax(iA, pA + (int64_t)iC * tR);
      iC += pC;
    }
  }
  int64_t xA = __shfl_up(iA, 1);
  uint32_t xC = __shfl_up(iC, 1);
  if (lane == 0) {
    xA = NEG;
    xC = 0;
  }
  const int64_t f0 = st->die_free[k];
  int64_t L = imax(xA, f0 + (int64_t)xC * tR);  // clock entering the lane's group
  uint32_t base = xC;
  if (lane == 63) {
    const int64_t Lend = imax(iA, f0 + (int64_t)iC * tR);
    totals[k] = iC;
    dfnew[k] = Lend;
    if (iC) {
      atomicMax((long long *)&ctl->max_dd, (long long)Lend);
      if (Lend >= TIME_LIMIT) atomicOr(&ctl->err, ERR_OVERFLOW);
    }
  }
  for (uint32_t t = ta; t < tb; t++) {
    tin_L[(size_t)t * K + k] = L;
    tin_base[(size_t)t * K + k] = base;
    const uint32_t c = agg_cnt[(size_t)t * K + k];
    if (c) L = imax(agg_A[(size_t)t * K + k], L + (int64_t)c * tR);
    base += c;
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
  uint32_t tot = block_excl_sum<WAVES>(s, &ex, sh);
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

// Pass 2 of the die stage.  Per chunk: stage the requests in (die queue,
// rank) order using the ranks pass 1 stored (LDS histogram + offsets, no
// re-ranking), compute exact die-done times with a segmented prefix max,
// and write them in die-queue order, filling the cell table on the way.
//
// Per die queue k the chunk needs a handful of numbers; they sit in two
// 16-byte records so that each phase reads one record per request (random
// k: one bank-conflicted access instead of several):
//   KA[k] = {koff: offset of k's run in the chunk, cnt: k's requests in the
//            tile before this chunk, L: die clock entering the chunk}
//   KW[k] = {rbase: die rank (within the call) of k's first request in the
//            chunk, pbase: its die-order position, lbo: k's column in the
//            cell table, tot: k's requests in the call}
// LDS: sval[CP] i64 | KA[K] | KW[K] | hist[K] u32 | (SC = 2) histA[K] u32 | refp[K] u32 |
//      skr [CP] u32 (key << 16 | rank in the step) | sloc [CP] u16, with CP = SC*CHUNK + SC*CHUNK/16
//
// SC pass-1 chunks are staged together (SC = 2 wherever its LDS fits: up to
// 954 die queues). A queue's run in die order then grows from one chunk's
// requests to two, so the die-order stores touch fewer partially written
// lines: measured 2.19 -> 1.83 ms on 2^28 requests over 512 queues.
template <int SC>
constexpr int chunk_pad() { return SC * CHUNK + SC * CHUNK / 16; }
// Pass 2 runs 1,024-thread blocks, 4 requests per thread per pass-1 chunk:
// with one chunk per step, measured 2.20 ms on 2^28 requests against
// 2.27 ms for two 512-thread blocks per CU.
constexpr int SBLK = 1024;
constexpr int SWAVES = SBLK / 64;
// Runs up to this length are scanned by one thread each; a chunk with a
// longer run (a hot die) takes the block-wide segmented scan.
constexpr uint32_t RUN_WALK_MAX = 64;

struct KeyA {
  uint32_t koff, cnt;
  int64_t L;
};
struct KeyW {
  uint32_t rbase, pbase, lbo, tot;
};

// REF (refresh quanta pending): the services depend on the call-wide rank,
// so the staged terms are issue - svc_sum(rank) and die_done =
// svc_sum(rank + 1) + prefix max; each admission that claims a quantum
// writes the quantum's completion (tR before its own read ends).
template <bool REF, int SC>
__global__ __launch_bounds__(SBLK) void k_die_scatter(
    const int64_t *__restrict__ issue, const uint32_t *__restrict__ KR, int64_t n, Geo g,
    int64_t tile_elems, const int64_t *__restrict__ tin_L, const uint32_t *__restrict__ tin_base,
    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ totals,
    int64_t *__restrict__ DD, uint32_t *__restrict__ IX, uint32_t *__restrict__ LB, uint32_t gmax,
    CallCtl *ctl, const DevState *st, uint64_t *__restrict__ WST, int64_t *__restrict__ ISS) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ SegMax shseg[SWAVES];
  __shared__ uint32_t shsum[SWAVES];
  __shared__ uint32_t s_nvalid, s_longrun;
  if (agent_load32(&ctl->err)) return;
  const uint32_t K = g.K;
  int64_t *sval = (int64_t *)smem;
  constexpr int SCH = SC * CHUNK;     // requests staged per step
  constexpr int CP = chunk_pad<SC>();
  constexpr int SITEMS = SCH / SBLK;  // per thread; the first SITEMS / SC come from the first chunk
  KeyA *KA = (KeyA *)(sval + CP);
  KeyW *KW = (KeyW *)(KA + K);
  uint32_t *hist = (uint32_t *)(KW + K);
  uint32_t *histA = hist + K;  // SC = 2: requests of each key in the first of the two chunks
  uint32_t *refp = histA + (SC == 2 ? K : 0);  // REF: pending quanta per key, read once per block
  uint32_t *skr = refp + K;
  uint16_t *sloc = (uint16_t *)(skr + CP);

  const uint32_t Dk = g.Dk;
  const size_t row = (size_t)blockIdx.x * K;
  // per-queue LDS records by LDS slot (lslot), as in pass 1, whose ranks
  // carry the slot
  for (uint32_t li = threadIdx.x; li < K; li += SBLK) {
    const uint32_t k = lkey(g, li);
    const uint32_t base = tin_base[row + k];  // die rank of the tile's first request of k
    KA[li] = KeyA{0u, 0u, tin_L[row + k]};
    const uint32_t ch = k / Dk;
    KW[li] = KeyW{base, seg_start[k] + base, ch * (gmax + 1) * Dk + (k - ch * Dk), totals[k]};
    if (REF) refp[li] = st->ref_pend[k];
  }
  const int64_t cbase = ctl->cbase;
  const uint32_t shift = ctl->shift, G = ctl->G;
  const bool narrow = shift <= 32;
  if (G) {  // clear the fused channel stage's look-back words of this call's cells (channel-major)
    const size_t nw = (size_t)G * g.C, step = (size_t)gridDim.x * SBLK;
    for (size_t q = (size_t)blockIdx.x * SBLK + threadIdx.x; q < nw; q += step) {
      const size_t c = q / G, at = c * gmax + (q - c * G);
      WST[at] = 0;
      WST[(size_t)gmax * g.C + at] = 0;
    }
  }
  const uint64_t relmask = narrow ? (uint64_t(1) << shift) - 1 : 0;
  const int64_t t0 = (int64_t)blockIdx.x * tile_elems;
  const int64_t t1 = imin(n, t0 + tile_elems);
  const uint32_t tR = (uint32_t)g.tR;

  // a chunk's requests are loaded while the previous one is scanned and
  // written (they are only needed up to the staging step)
  int64_t iss[SITEMS];
  uint32_t kr[SITEMS];
  auto fetch = [&](int64_t cc) {
#pragma unroll
    for (int e = 0; e < SITEMS; e++) {
      const int64_t i = cc + e * SBLK + threadIdx.x;
      iss[e] = 0;
      kr[e] = (uint32_t)KEY_NONE << 16;
      if (i < t1) {
        iss[e] = issue[i];
        kr[e] = KR[i];
      }
    }
  };
  if (t0 < t1) fetch(t0);
  for (int64_t c0 = t0; c0 < t1; c0 += SCH) {
    for (uint32_t k = threadIdx.x; k < K; k += SBLK) {
      hist[k] = 0;
      if (SC == 2) histA[k] = 0;
    }
    if (threadIdx.x == 0) s_longrun = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < SITEMS; e++) {
      const uint32_t k = kr[e] >> 16;
      if (k != KEY_NONE) atomicAdd(SC == 2 && e < SITEMS / 2 ? &histA[k] : &hist[k], 1u);
    }
    __syncthreads();
    {  // chunk offsets of each key's run
      const uint32_t per = (K + SBLK - 1) / SBLK;
      const uint32_t a0 = threadIdx.x * per, b0 = min(K, a0 + per);
      uint32_t sum = 0;
      for (uint32_t k = a0; k < b0; k++) {
        if (SC == 2) hist[k] += histA[k];
        sum += hist[k];
      }
      uint32_t ex;
      const uint32_t all = block_excl_sum<SWAVES>(sum, &ex, shsum);
      uint32_t longest = 0;
      for (uint32_t k = a0; k < b0; k++) {
        KA[k].koff = ex;
        ex += hist[k];
        longest = max(longest, hist[k]);
      }
      if (threadIdx.x == 0) s_nvalid = all;
      if (longest > RUN_WALK_MAX) s_longrun = 1u;
    }
    __syncthreads();
    // stage v = issue - r0*tR in die order (r0 = rank of the request among
    // k's in the tile); a run's head also folds in the entering clock,
    // M_k = L_k - cnt_k*tR, so the segmented prefix max below is the whole
    // Lindley term: die_done = (r0+1)*tR + max(M_k, max of v over the run)
#pragma unroll
    for (int e = 0; e < SITEMS; e++) {
      const uint32_t k = kr[e] >> 16;
      if (k != KEY_NONE) {
        const KeyA ka = KA[k];
        // pass 1's rank is within its own chunk: the second chunk's requests
        // of k follow the first chunk's
        const uint32_t rc = (kr[e] & 0xFFFFu) + (SC == 2 && e >= SITEMS / 2 ? histA[k] : 0u);
        const uint32_t P = pad16(ka.koff + rc);
        int64_t v;
        if (REF) {
          const uint32_t R = refp[k], g0 = KW[k].rbase;
          v = iss[e] - svc_sum(g0 + rc, R, g.tR, g.tQ);
          if (rc == 0) v = imax(v, ka.L - svc_sum(g0, R, g.tR, g.tQ));
        } else {
          v = iss[e] - (int64_t)mul32(ka.cnt + rc, tR);
          if (rc == 0) v = imax(v, ka.L - (int64_t)mul32(ka.cnt, tR));
        }
        sval[P] = v;
        skr[P] = k << 16 | rc;
        sloc[P] = (uint16_t)(e * SBLK + threadIdx.x);
        if (ISS) {  // register blocking: the issue times in die order as well
          const uint32_t gp = KW[k].pbase + rc;
          if (gp < n) ISS[gp] = iss[e];
        }
      }
    }
    __syncthreads();
    if (c0 + SCH < t1) fetch(c0 + SCH);
    const uint32_t nv = s_nvalid;
    if (!s_longrun) {
      // one thread per die queue walks its run with a running maximum (the
      // run's head already holds the entering clock)
      for (uint32_t k = threadIdx.x; k < K; k += SBLK) {
        const uint32_t t = hist[k];
        if (!t) continue;
        const KeyA ka = KA[k];
        int64_t run = NEG;
        if (REF) {
          const uint32_t R = refp[k], g0 = KW[k].rbase;
          for (uint32_t q = 0; q < t; q++) {
            const uint32_t P = pad16(ka.koff + q);
            run = imax(run, sval[P]);
            sval[P] = svc_sum(g0 + q + 1, R, g.tR, g.tQ) + run;
          }
          continue;
        }
        for (uint32_t q = 0; q < t; q++) {
          const uint32_t P = pad16(ka.koff + q);
          run = imax(run, sval[P]);
          sval[P] = (int64_t)mul32(ka.cnt + q + 1, tR) + run;
        }
      }
    } else {  // a long run: segmented scan over the whole block
      const uint32_t p0 = threadIdx.x * SITEMS;
      int64_t vals[SITEMS];
      SegMax agg = {0, NEG};
#pragma unroll
      for (int q = 0; q < SITEMS; q++) {
        const uint32_t p = p0 + q;
        vals[q] = NEG;
        if (p < nv) {
          const int64_t v = sval[pad16(p)];
          vals[q] = v;
          agg = seg_comb(agg, SegMax{(skr[pad16(p)] & 0xFFFFu) == 0, v});
        }
      }
      SegMax ex = block_excl_segmax<SWAVES>(agg, shseg);
      int64_t run = ex.v;  // prefix of the segment continuing into this thread
#pragma unroll
      for (int q = 0; q < SITEMS; q++) {
        const uint32_t p = p0 + q;
        if (p < nv) {
          const uint32_t kr2 = skr[pad16(p)];
          const uint32_t rc = kr2 & 0xFFFFu;
          run = (rc == 0) ? vals[q] : imax(run, vals[q]);
          const uint32_t kk = kr2 >> 16;
          if (REF)
            sval[pad16(p)] = svc_sum(KW[kk].rbase + rc + 1, refp[kk], g.tR, g.tQ) + run;
          else
            sval[pad16(p)] = (int64_t)mul32(KA[kk].cnt + rc + 1, tR) + run;
        }
      }
    }
    __syncthreads();
    // write die-ordered (die_done, index); fill the cell table
    for (uint32_t p = threadIdx.x; p < nv; p += SBLK) {
      const uint32_t P = pad16(p);
      const uint32_t kr2 = skr[P];
      const uint32_t k = kr2 >> 16;
      const uint32_t rc = kr2 & 0xFFFFu;
      const KeyW kw = KW[k];
      const uint32_t r = kw.rbase + rc;  // die rank within this call
      const int64_t dd = sval[P];
      const uint32_t gpos = kw.pbase + rc;
      if (gpos < n) {
        const uint32_t ix = (uint32_t)(c0 + sloc[P]);
        if (narrow)  // one word: offset of die-done in its cell, request index
          reinterpret_cast<uint64_t *>(DD)[gpos] = ((uint64_t)(dd - cbase) & relmask) << 32 | ix;
        else {
          DD[gpos] = dd;
          IX[gpos] = ix;
        }
      }
      if (REF && r < refp[k]) {  // this admission claimed quantum r of its queue's pending ones
        const uint32_t kq = lkey(g, k);
        *st->ref_slot[st->ref_off[kq] + st->ref_head[kq] + r] = dd - g.tR;
      }
      // die-done of slot p - 1 (the same queue's previous request when rc > 0):
      // lane l - 1's value, or read back by lane 0
      int64_t pdd = dpp64<DPP_WAVE_SHR1, 0xF>(dd, dd);
      if (lane_id() == 0 && p > 0) pdd = sval[pad16(p - 1)];
      const int64_t prev = (rc > 0) ? pdd : KA[k].L;
      const int64_t cell = imin((dd - cbase) >> shift, (int64_t)G);
      const int64_t pcell = (r == 0) ? -1 : imin((prev - cbase) >> shift, (int64_t)G);
      uint32_t *lbrow = LB + kw.lbo;
      for (int64_t c = pcell + 1; c <= cell; c++) lbrow[(size_t)c * Dk] = r;
      if (r + 1 == kw.tot)
        for (int64_t c = cell + 1; c <= (int64_t)G; c++) lbrow[(size_t)c * Dk] = r + 1;
    }
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < K; k += SBLK) {
      const uint32_t t = hist[k];
      if (t) {
        KA[k].L = sval[pad16(KA[k].koff + t - 1)];
        KA[k].cnt += t;
        KW[k].rbase += t;
        KW[k].pbase += t;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ channel stage

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


constexpr int CAP_S = 256;     // requests per round of a streamed cell
constexpr int SLOTS_MAX = 16;  // die runs per channel on the bucket path

struct CellLds {
  union {
    struct {
      uint64_t in[MCAP];                 // (dd - cell start) << 32 | index, in run order
      uint8_t tbl[MAX_BUCKETS][SLOTS_MAX];  // 1 + position in its run of die d's request in bucket q
    } f;
    struct {
      int64_t dd[2][CAP_S];
      uint32_t ix[2][CAP_S];
      uint8_t tg[2][CAP_S];
    } s;
  } u;
  uint32_t rb[MAX_RUNS + 1]; // run offsets in the staging buffer
  uint32_t lo[MAX_RUNS];     // run bounds: global positions in the die order
  uint32_t hi[MAX_RUNS];
  uint32_t cur[MAX_RUNS];
  uint32_t take[MAX_RUNS];
  uint32_t used[MAX_RUNS];
  uint32_t safe;
};

// Sort keys of the bucket path are integers below 2^51 held in the mantissa
// of a double in [1, 2) (exponent bits 0x3FF): there IEEE order is integer
// order, so one exact v_min_f64 / v_max_f64 pair is a whole compare-exchange.
constexpr uint64_t KEY_ONE = uint64_t(0x3FF) << 52;
constexpr uint64_t KEY_EMPTY = KEY_ONE | ((uint64_t(1) << 52) - 1);  // above every key

DEVI void cx_key(uint64_t &lo, uint64_t &hi) {
  const double a = __builtin_bit_cast(double, lo), b = __builtin_bit_cast(double, hi);
  double mn, mx;
  asm("v_min_f64 %0, %1, %2" : "=v"(mn) : "v"(a), "v"(b));
  asm("v_max_f64 %0, %1, %2" : "=v"(mx) : "v"(a), "v"(b));
  lo = __builtin_bit_cast(uint64_t, mn);
  hi = __builtin_bit_cast(uint64_t, mx);
}

// Batcher's odd-even merge sort over SL registers (SL a power of two; 63
// compare-exchanges for 16), ascending.
template <int SL>
DEVI void sort_slots(uint64_t (&a)[SL]) {
#pragma unroll
  for (int p = 1; p < SL; p <<= 1) {
#pragma unroll
    for (int k = p; k >= 1; k >>= 1) {
#pragma unroll
      for (int j = k % p; j + k < SL; j += 2 * k) {
#pragma unroll
        for (int i = 0; i < k; i++) {
          if (i + j + k < SL && (i + j) / (2 * p) == (i + j + k) / (2 * p)) cx_key(a[i + j], a[i + j + k]);
        }
      }
    }
  }
}

// One wave streams a cell through the LDS in rounds of at most CAP_S
// requests (cells that are too wide or too full for the bucket path).  Each
// round loads at most CAP_S/R requests per run, ranks them (binary searches
// in the other runs), and serves the prefix that no unloaded request can
// precede.  gacc: running channel term; returns it after the cell.
DEVI int64_t stream_cell(CellLds &S, const int64_t *DD, const uint32_t *IX, bool narrow, int64_t cstart,
                         int R, int64_t gacc, int64_t rank0, int64_t xfer, bool emit, int64_t *complete,
                         uint32_t n, uint32_t *errb) {
  const uint32_t lane = lane_id();
  if (lane < (uint32_t)R) S.cur[lane] = S.lo[lane];
  wave_sync();
  int64_t done = 0;
  const uint32_t quota = CAP_S / R;
  while (true) {
    uint32_t rem = 0, take = 0;
    if (lane < (uint32_t)R) rem = S.hi[lane] - S.cur[lane];
    const uint32_t tot = wave_sum(rem);
    if (tot == 0) break;
    take = tot <= (uint32_t)CAP_S ? rem : min(rem, quota);
    const uint32_t rbx = wave_excl_sum(take);
    const uint32_t m = wave_sum(take);
    if (lane < (uint32_t)R) {
      S.rb[lane] = rbx;
      S.take[lane] = take;
      S.used[lane] = 0;
    }
    if (lane == 0) S.rb[R] = m;
    wave_sync();
    for (uint32_t p = lane; p < m; p += 64) {
      const int d = run_of(S.rb, R, p);
      const uint32_t src = S.cur[d] + (p - S.rb[d]);
      if (narrow) {
        const uint64_t x = reinterpret_cast<const uint64_t *>(DD)[src];
        S.u.s.dd[0][p] = cstart + (int64_t)(x >> 32);
        S.u.s.ix[0][p] = (uint32_t)x;
      } else {
        S.u.s.dd[0][p] = DD[src];
        S.u.s.ix[0][p] = IX[src];
      }
      S.u.s.tg[0][p] = (uint8_t)d;
    }
    wave_sync();
    // merged order: own index + requests of the other runs that precede
    for (uint32_t p = lane; p < m; p += 64) {
      const int d = S.u.s.tg[0][p];
      const int64_t x = S.u.s.dd[0][p];
      const uint32_t xi = S.u.s.ix[0][p];
      uint32_t r = p - S.rb[d];
      for (int d2 = 0; d2 < R; d2++) {
        if (d2 == d) continue;
        uint32_t a = S.rb[d2], b = S.rb[d2 + 1];
        while (a < b) {
          const uint32_t mid = (a + b) >> 1;
          if (key_less(S.u.s.dd[0][mid], S.u.s.ix[0][mid], x, xi)) a = mid + 1;
          else b = mid;
        }
        r += a - S.rb[d2];
      }
      S.u.s.dd[1][r] = x;
      S.u.s.ix[1][r] = xi;
      S.u.s.tg[1][r] = (uint8_t)d;
    }
    wave_sync();
    // safe prefix: everything up to the smallest last-loaded request of a
    // run that still has requests behind it
    if (lane == 0) {
      bool ok = false;
      int64_t vd = 0;
      uint32_t vi = 0;
      for (int d = 0; d < R; d++) {
        const uint32_t t = S.take[d];
        if (t > 0 && t < S.hi[d] - S.cur[d]) {
          const uint32_t q = S.rb[d] + t - 1;
          if (!ok || key_less(S.u.s.dd[0][q], S.u.s.ix[0][q], vd, vi)) {
            vd = S.u.s.dd[0][q];
            vi = S.u.s.ix[0][q];
            ok = true;
          }
        }
      }
      uint32_t safe = m;
      if (ok) {
        uint32_t a = 0, b = m;
        while (a < b) {
          const uint32_t mid = (a + b) >> 1;
          if (!key_less(vd, vi, S.u.s.dd[1][mid], S.u.s.ix[1][mid])) a = mid + 1;
          else b = mid;
        }
        safe = a;
      }
      S.safe = safe;
    }
    wave_sync();
    const uint32_t safe = S.safe;
    for (uint32_t base = 0; base < safe; base += 64) {
      const uint32_t p = base + lane;
      int64_t v = NEG;
      if (p < safe) {
        v = S.u.s.dd[1][p] - (rank0 + done + p) * xfer;
        atomicAdd(&S.used[S.u.s.tg[1][p]], 1u);
      }
      const int64_t q = imax(gacc, wave_incl_max(v));
      if (emit && p < safe) {
        const int64_t cpl = (rank0 + done + p + 1) * xfer + q;
        if (cpl >= TIME_LIMIT) *errb |= ERR_OVERFLOW;
        const uint32_t ix = S.u.s.ix[1][p];
        if (ix < n) complete[ix] = cpl;
      }
      gacc = imax(gacc, wave_max(v));
    }
    done += safe;
    wave_sync();
    if (lane < (uint32_t)R) S.cur[lane] += S.used[lane];
    wave_sync();
  }
  return gacc;
}

// Channel stage.  With channel ranks k (1-based) and the channel free at f0
// before the call, complete_k = k*xfer + max(f0, max_{i<=k} (dd_(i) - (i-1)*xfer)).
// A cell knows its first rank from the cell table (the sum of its row), so
// its aggregate is one number, M_j = max over its requests of
// (dd - (rank-1)*xfer), and the term entering cell j is max(f0, M_j' for
// j' < j).  On the bucket path k_cell_chan merges each cell once and finds
// the entering term by a look-back over earlier windows.  Grids off the
// bucket path run reduce, scan, reduce again:
//   k_cell_agg   M_j of every cell;
//   k_cell_scan  per channel, the running maximum of M_j seeded with f0;
//   k_cell_rest  every cell again, now writing complete[] with its term.
//
// One wave per cell.  The bucket path (buckets of width 2^lg_tR <= tR hold
// at most one request per die): lane q gathers the requests of bucket q --
// die d's is at 1 + the byte the LDS table holds for (q, d) -- sorts them
// in registers, and owns merged positions boff..boff+cnt-1 of the cell.
// Cells that are too wide or too full stream through the LDS instead.

// Cell of iteration `it` of this block: (window, channel) order,
// grid-stride, so all blocks move along one common time front.
DEVI bool cell_at(uint32_t it, uint32_t N, uint32_t C, uint32_t G, uint32_t &c, uint32_t &j) {
  const uint64_t cell = (uint64_t)blockIdx.x + (uint64_t)it * gridDim.x;
  if (cell >= N) return false;
  j = (uint32_t)cell / C;
  c = (uint32_t)cell - j * C;
  return true;
}

// One pass over cell (c, j).  Returns M_j; with EMIT, writes instead the
// completion of each of its requests given the entering term gin.
// A cell's runs, lane d = die run d: die-order bounds [lo, hi) and the die
// rank r0 of the first one.
struct CellRuns {
  uint32_t lo, hi, r0;
};
DEVI CellRuns cell_runs(const uint32_t *__restrict__ LB, const uint32_t *__restrict__ seg_start,
                        const uint32_t *__restrict__ totals, uint32_t Dk, uint32_t gmax, uint32_t c,
                        uint32_t j) {
  CellRuns r = {0, 0, 0};
  const uint32_t lane = lane_id();
  if (lane < Dk) {
    const uint32_t k = c * Dk + lane;
    if (totals[k] != 0) {
      const uint32_t *lbrow = LB + (size_t)c * (gmax + 1) * Dk + lane;
      const uint32_t sg = seg_start[k];
      r.r0 = lbrow[(size_t)j * Dk];
      r.lo = r.r0 + sg;
      r.hi = lbrow[(size_t)(j + 1) * Dk] + sg;
    }
  }
  return r;
}

// The bucket path's loads: lane q < 64 reads entry q of every run (runs of
// bucketable cells hold at most 64), all in flight at once.
template <int SL>
DEVI void load_runs(const int64_t *__restrict__ DD, const CellRuns &cr, int R, uint64_t (&xv)[SL]) {
  const uint32_t lane = lane_id();
  const uint64_t *DX = reinterpret_cast<const uint64_t *>(DD);
  const uint32_t len = cr.hi - cr.lo;
#pragma unroll
  for (int d = 0; d < SL; d++) {
    const uint32_t lod = __builtin_amdgcn_readlane(cr.lo, d);
    const uint32_t lend = __builtin_amdgcn_readlane(len, d);
    xv[d] = 0;
    if (d < R && lane < lend) xv[d] = DX[lod + lane];
  }
}

// Whether the cell grid allows the bucket path at all: buckets of width
// 2^lg_tR, at most 64 of them per cell, packed 32-bit cell offsets, and at
// most SL die runs per channel.  A cell then takes it if no run holds more
// than 64 of its requests.
template <int SL>
DEVI bool grid_bucketable(const Geo &g, uint32_t shift) {
  return (shift - g.lg_tR <= 6) && shift <= 32 && g.lg_tR <= 20 && (int)g.Dk <= SL;
}

template <int SL, bool EMIT>
DEVI int64_t cell_pass(CellLds &S, const int64_t *__restrict__ DD, const uint32_t *__restrict__ IX,
                       const CellRuns &cr, const uint64_t (&xv)[SL], const Geo &g, uint32_t shift,
                       int64_t cbase, uint32_t j, int64_t gin, int64_t *complete, uint32_t n,
                       uint32_t *errb) {
  const uint32_t lane = lane_id();
  const uint32_t Dk = g.Dk;
  const uint32_t lgt = g.lg_tR;
  const bool bucketable = grid_bucketable<SL>(g, shift);
  const int R = (int)Dk;
  const int64_t xfer = g.xfer;
  const int64_t cstart = cbase + ((int64_t)j << shift);
  const uint32_t lo = cr.lo, hi = cr.hi, r0 = cr.r0;
  const uint32_t len = hi - lo;
  const uint32_t rbx = wave_excl_sum(len);
  const uint32_t m = wave_sum(len);
  const int64_t rank0 = wave_sum(r0);  // channel rank of the cell's first request
  if (m == 0) return NEG;
  if (lane < Dk) {
    S.lo[lane] = lo;
    S.hi[lane] = hi;
    S.rb[lane] = rbx;
  }
  if (lane == 0) S.rb[R] = m;
  wave_sync();
  const uint32_t maxlen = wave_umax(lane < Dk ? len : 0u);
  if (!(bucketable && maxlen <= 64)) {
    if (EMIT) {
      stream_cell(S, DD, IX, shift <= 32, cstart, R, gin, rank0, xfer, true, complete, n, errb);
      return NEG;
    }
    return stream_cell(S, DD, IX, shift <= 32, cstart, R, NEG, rank0, xfer, false, complete, n, errb);
  }
  uint64_t slot[SL];
  uint32_t cnt = 0;
  // clear the bucket table (1 KB: 16 B per lane)
  reinterpret_cast<uint4 *>(&S.u.f.tbl[0][0])[lane] = make_uint4(0, 0, 0, 0);
  // the runs were loaded by load_runs.  Bucketable cells are at most 2^32 ns
  // wide, so their entries are packed words (offset in the cell << 32 |
  // index); staged as the bucket's sort key: offset in the bucket (< 2^20)
  // << 31 | index.
  wave_sync();
  const uint64_t offmask = (uint64_t(1) << lgt) - 1;
#pragma unroll
  for (int d = 0; d < SL; d++) {
    const uint32_t lend = __builtin_amdgcn_readlane(len, d);
    const uint32_t rbd = __builtin_amdgcn_readlane(rbx, d);
    if (d < R && lane < lend) {
      const uint64_t rel = xv[d] >> 32;
      S.u.f.in[rbd + lane] = KEY_ONE | (rel & offmask) << 31 | (xv[d] & 0xFFFFFFFFull);
      S.u.f.tbl[rel >> lgt][d] = (uint8_t)(lane + 1);
    }
  }
  wave_sync();
  // lane q: gather, sort and count bucket q
  {
    const uint4 row = reinterpret_cast<const uint4 *>(&S.u.f.tbl[0][0])[lane];
    const uint32_t rw[4] = {row.x, row.y, row.z, row.w};
#pragma unroll
    for (int d = 0; d < SL; d++) {
      const uint32_t y = (rw[d >> 2] >> (8 * (d & 3))) & 0xFFu;
      const uint32_t rbd = __builtin_amdgcn_readlane(rbx, d);
      slot[d] = KEY_EMPTY;
      if (y) {
        slot[d] = S.u.f.in[rbd + y - 1];
        cnt++;
      }
    }
  }
  sort_slots<SL>(slot);
  const uint32_t boff = wave_excl_sum(cnt);
  // Lindley prefix over the merged order, in registers: merged position p
  // has value dd - (rank0 + p) * xfer, dd = cell start + bucket start + offset
  const int64_t cst = cstart + ((int64_t)lane << lgt) - rank0 * xfer;
  int64_t loc = NEG;
#pragma unroll
  for (int i = 0; i < SL; i++) {
    if ((uint32_t)i < cnt) {
      const int64_t v = cst + (int64_t)((slot[i] >> 31) & 0x1FFFFFu) - (int64_t)mul32(boff + i, (uint32_t)xfer);
      loc = imax(loc, v);
    }
  }
  if (!EMIT) return wave_max(loc);
  int64_t carry = __shfl_up(wave_incl_max(loc), 1);
  if (lane == 0) carry = NEG;
  carry = imax(carry, gin);
  const int64_t r0x = rank0 * xfer;
#pragma unroll
  for (int i = 0; i < SL; i++) {
    if ((uint32_t)i < cnt) {
      const int64_t v = cst + (int64_t)((slot[i] >> 31) & 0x1FFFFFu) - (int64_t)mul32(boff + i, (uint32_t)xfer);
      carry = imax(carry, v);
      const int64_t cpl = r0x + (int64_t)mul32(boff + i + 1, (uint32_t)xfer) + carry;
      if (cpl >= TIME_LIMIT) *errb |= ERR_OVERFLOW;
      const uint32_t ix = (uint32_t)slot[i] & 0x7FFFFFFFu;
      if (ix < n) complete[ix] = cpl;
    }
  }
  return NEG;
}

// The cell loop of both passes.  (Loading the next cell's runs while the
// current one merges needs a second set of run registers: it halved the
// occupancy of the aggregate pass and measured slower in the output pass.)
template <int SL, typename Body>
DEVI void cell_loop(const int64_t *__restrict__ DD, const uint32_t *__restrict__ LB,
                    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ totals, const Geo &g,
                    uint32_t gmax, uint32_t N, uint32_t G, Body body) {
  uint32_t c, j;
  for (uint32_t it = 0; cell_at(it, N, g.C, G, c, j); it++) {
    const CellRuns cr = cell_runs(LB, seg_start, totals, g.Dk, gmax, c, j);
    uint64_t xv[SL];
    load_runs<SL>(DD, cr, (int)g.Dk, xv);
    body(c, j, cr, xv);
    wave_sync();
  }
}

constexpr uint32_t CMIN_NONE = 0xFFFFFFFFu;

// Grids off the bucket path (cells too wide for 64 buckets, or more die
// queues per channel than SL): M_j of every cell, which is listed for
// k_cell_rest.  On the bucket path k_cell_chan does the whole stage and
// this kernel returns at once.
template <int SL>
__global__ __launch_bounds__(64) void k_cell_agg(
    const int64_t *__restrict__ DD, const uint32_t *__restrict__ IX, const uint32_t *__restrict__ LB,
    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ totals, Geo g,
    CallCtl *ctl, int64_t *__restrict__ AGG, uint32_t *__restrict__ NBL, uint32_t gmax, uint32_t n) {
  extern __shared__ __align__(16) unsigned char smem[];
  CellLds &S = *(CellLds *)smem;
  if (agent_load32(&ctl->err)) return;
  const uint32_t G = ctl->G, N = G * g.C, shift = ctl->shift;
  if (grid_bucketable<SL>(g, shift)) return;
  const int64_t cbase = ctl->cbase;
  uint32_t errb = 0;
  cell_loop<SL>(DD, LB, seg_start, totals, g, gmax, N, G,
                [&](uint32_t c, uint32_t j, const CellRuns &cr, const uint64_t (&xv)[SL]) {
                  const int64_t M = cell_pass<SL, false>(S, DD, IX, cr, xv, g, shift, cbase, j, NEG,
                                                         nullptr, n, &errb);
                  const uint32_t m = wave_sum(cr.hi - cr.lo);
                  if (lane_id() == 0) {
                    AGG[(size_t)c * gmax + j] = M;
                    if (m > 0) NBL[atomicAdd(&ctl->n_rest, 1u)] = j * g.C + c;
                  }
                });
  if (errb) atomicOr(&ctl->err, errb);
}

// Per channel: GIN[j] = max(f0, M_j' for j' < j); the channel clock after the
// call is (its request count) * xfer + max(f0, every M_j).  One block per
// channel, each thread a contiguous range of windows: fold, block scan, walk.
__global__ __launch_bounds__(BLK) void k_cell_scan(const int64_t *__restrict__ AGG, int64_t *__restrict__ GIN,
                                                   const uint32_t *__restrict__ totals, Geo g,
                                                   CallCtl *ctl, const DevState *st,
                                                   int64_t *__restrict__ cfnew, uint32_t gmax) {
  __shared__ int64_t sh[WAVES];
  if (agent_load32(&ctl->err)) return;
  if (grid_bucketable<SLOTS_MAX>(g, ctl->shift)) return;  // the bucket path is k_cell_chan's
  const uint32_t c = blockIdx.x, G = ctl->G;
  const size_t row = (size_t)c * gmax;
  const uint32_t per = (G + BLK - 1) / BLK;
  const uint32_t ja = min(G, threadIdx.x * per), jb = min(G, ja + per);
  int64_t m = NEG;
  for (uint32_t j = ja; j < jb; j++) m = imax(m, AGG[row + j]);
  const int64_t ex = block_excl_max<WAVES>(m, sh);
  const int64_t f0 = st->chan_free[c];
  int64_t carry = imax(f0, ex);
  for (uint32_t j = ja; j < jb; j++) {
    GIN[row + j] = carry;
    carry = imax(carry, AGG[row + j]);
  }
  if (threadIdx.x == BLK - 1) {
    uint64_t tot = 0;
    for (uint32_t d = 0; d < g.Dk; d++) tot += totals[c * g.Dk + d];
    const int64_t last = (int64_t)tot * g.xfer + imax(f0, imax(ex, m));
    cfnew[c] = last;
    // the channel's last completion of this call
    if (tot) atomicMax((long long *)&ctl->max_cpl, (long long)last);
  }
}

// ---- Fused channel stage (grids on the bucket path).  The work is cut into
// units: a unit is one time window j and a group of up to CH_GROUP channels
// (all of them when C <= CH_GROUP), and units are claimed in (window, group)
// order from a counter of the call.  One 1,024-thread workgroup per unit:
//   1. each wave merges two of the unit's cells (bucket path, kept in
//      registers) and publishes each cell's term M_j;
//   2. per channel, the term entering the cell, max(f0, M_j' for j' < j),
//      by a decoupled look-back over the earlier windows' published words:
//      the nearest inclusive term plus the aggregates in between;
//   3. it publishes the inclusive term max(entering, M_j);
//   4. it writes the completions.  Those of one window fall in a band of
//      request indices (each die queue serves its next requests), so each
//      completion is staged in LDS at its index's offset from the band start
//      as a 32-bit offset from a base, and the band is written in index
//      order (whole lines); completions outside the staged span, or whose
//      offset does not fit, are stored directly.
// A unit waits only for units claimed before it: their workgroups are
// running and publish their aggregates without waiting, so every wait ends.
// The wait is bounded all the same; running past the bound fails the call
// with ERR_INTERNAL instead of hanging.  The published words are single
// 64-bit atomics that carry their own validity (0 = not yet), cleared by
// k_die_scatter for the cells of the call and laid out channel-major, so a
// half-wave polling 32 consecutive windows of one channel reads two lines.
constexpr int WIN_WAVES = 16;
constexpr int WIN_THREADS = WIN_WAVES * 64;
constexpr int CH_GROUP = 2 * WIN_WAVES;
constexpr uint32_t WIN_SLOTS = 32768;
constexpr uint32_t WIN_EMPTY = 0xFFFFFFFFu;
constexpr uint32_t LOOKBACK_ROUNDS = 1u << 22;

struct WinLds {
  uint32_t stage[WIN_SLOTS];                         // completion - wbase at index lo + slot
  uint8_t tbl[WIN_WAVES][MAX_BUCKETS][SLOTS_MAX];   // per wave: 1 + position in run d of bucket q's entry
  uint32_t rmin[WIN_WAVES];
  int64_t rbase[WIN_WAVES];
  uint32_t top;                                      // staged slots in use
  uint32_t unit;
};

// Stage slot of band offset r.  One channel's requests often sit at a
// fixed stride in the index space (sequential streams stripe over the
// channels), so the offsets one store instruction writes can share their
// low bits; XOR-ing in the next six bits spreads them over the LDS banks,
// while each aligned group of 64 consecutive offsets stays a permutation of
// itself (the write-out reads them conflict-free).
DEVI uint32_t win_slot(uint32_t r) { return r ^ ((r >> 6) & 63u); }

DEVI uint32_t wave_umin(uint32_t x) { return ~wave_umax(~x); }
DEVI int64_t wave_min(int64_t x) { return -wave_max(-x); }

// Look-back words: 0 = not yet published, else the value + 2^62 (every
// published value lies in [NEG, 2^62)).
DEVI uint64_t enc_time(int64_t x) { return (uint64_t)x + (uint64_t(1) << 62); }
DEVI int64_t dec_time(uint64_t w) { return (int64_t)(w - (uint64_t(1) << 62)); }
DEVI uint64_t agent_load64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEVI void agent_store64(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inclusive maximum within each half (32 lanes) of the wave: lanes 31 and
// 63 end up holding the two halves' maxima.
DEVI int64_t half_incl_max(int64_t x) {
  x = imax(x, dpp64<DPP_ROW_SHR1, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR2, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR4, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR8, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_BCAST15, 0xA>(NEG, x));
  return x;
}
DEVI int64_t lane_i64(int64_t x, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)x >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// The terms entering window j of two channels, one per half-wave (lanes
// 0-31: channel ca, 32-63: channel cb; a channel >= C is skipped).  Lane s
// of a half inspects window base - s: its inclusive word, else its
// aggregate.  A round ends at the nearest inclusive word (or before window
// 0, where the term is the channel's clock f0) if no aggregate before it is
// missing; otherwise the half folds what precedes the first missing one and
// polls again from there.
DEVI void look_back2(const uint64_t *WAGG, const uint64_t *WINC, uint32_t C, uint32_t gmax, uint32_t j,
                     uint32_t ca, uint32_t cb, int64_t f0a, int64_t f0b, int64_t &ga, int64_t &gb,
                     uint32_t *errb) {
  const uint32_t lane = lane_id(), s = lane & 31;
  const bool hi = lane >= 32;
  const uint32_t c = hi ? cb : ca;
  const int64_t f0 = hi ? f0b : f0a;
  int64_t acc0 = NEG, acc1 = NEG;
  int64_t base0 = (int64_t)j - 1, base1 = (int64_t)j - 1;
  bool done0 = ca >= C, done1 = cb >= C;
  uint32_t rounds = 0;
  while (!(done0 && done1)) {
    const bool mine_done = hi ? done1 : done0;
    const int64_t jj = (hi ? base1 : base0) - (int64_t)s;
    int stt = 2;  // 2: inclusive (or nothing left to fold), 1: aggregate, 0: not yet published
    int64_t v = NEG;
    if (!mine_done) {
      if (jj < 0) {
        v = f0;
      } else {
        const size_t at = (size_t)c * gmax + (size_t)jj;  // a half reads 32 consecutive words
        const uint64_t wi = agent_load64(&WINC[at]);
        if (wi) {
          v = dec_time(wi);
        } else {
          const uint64_t wa = agent_load64(&WAGG[at]);
          stt = wa ? 1 : 0;
          if (wa) v = dec_time(wa);
        }
      }
    }
    const uint64_t incl = __ballot(stt == 2), none = __ballot(stt == 0);
    const uint32_t bi0 = (uint32_t)incl, bi1 = (uint32_t)(incl >> 32);
    const uint32_t bn0 = (uint32_t)none, bn1 = (uint32_t)(none >> 32);
    const uint32_t fi0 = bi0 ? (uint32_t)__builtin_ctz(bi0) : 32u, fi1 = bi1 ? (uint32_t)__builtin_ctz(bi1) : 32u;
    const uint32_t fn0 = bn0 ? (uint32_t)__builtin_ctz(bn0) : 32u, fn1 = bn1 ? (uint32_t)__builtin_ctz(bn1) : 32u;
    // fold: through the inclusive word if it precedes every gap, else up to the gap
    const uint32_t fi = hi ? fi1 : fi0, fn = hi ? fn1 : fn0;
    const uint32_t lim = (fi < fn) ? fi + 1 : fn;
    const int64_t red = half_incl_max(s < lim ? v : NEG);
    bool stalled = false;
    if (!done0) {
      acc0 = imax(acc0, lane_i64(red, 31));
      if (fi0 < fn0) done0 = true;
      else {
        base0 -= fn0;
        stalled |= fn0 == 0;
      }
    }
    if (!done1) {
      acc1 = imax(acc1, lane_i64(red, 63));
      if (fi1 < fn1) done1 = true;
      else {
        base1 -= fn1;
        stalled |= fn1 == 0;
      }
    }
    if (stalled) {
      if (++rounds > LOOKBACK_ROUNDS) {
        *errb |= ERR_INTERNAL;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  ga = acc0;
  gb = acc1;
}

// A merged cell, held in registers: lane q owns bucket q's entries, sorted
// (slot), their count and first merged position; plus the cell's size, its
// smallest request index, the channel rank of its first request, and per
// lane the maximum of dd - (rank0 + position) * xfer over its entries.
template <int SL>
struct Merged {
  uint64_t slot[SL];
  uint32_t cnt, boff;
  uint32_t m, head;
  int64_t rank0, loc;
};

// Merge one bucketable cell (lane q gathers bucket q's entries from the
// lanes that loaded them, sorts them, and takes merged positions
// boff..boff+cnt-1).  Its run of die d holds at most one entry per bucket.
template <int SL>
DEVI void cell_merge(uint8_t (*tbl)[SLOTS_MAX], const CellRuns &cr, const uint64_t (&xv)[SL], const Geo &g,
                     int64_t cstart, Merged<SL> &M, uint32_t *errb) {
  const uint32_t lane = lane_id();
  const int R = (int)g.Dk;
  const uint32_t lgt = g.lg_tR;
  const int64_t xfer = g.xfer;
  const uint32_t len = cr.hi - cr.lo;
  M.m = wave_sum(len);
  M.cnt = 0;
  M.boff = 0;
  M.head = CMIN_NONE;
  M.rank0 = 0;
  M.loc = NEG;
#pragma unroll
  for (int d = 0; d < SL; d++) M.slot[d] = KEY_EMPTY;
  if (M.m == 0) return;
  if (wave_umax(lane < (uint32_t)R ? len : 0u) > 64) {  // impossible on a bucketable grid
    *errb |= ERR_INTERNAL;
    M.m = 0;
    return;
  }
  M.rank0 = wave_sum(cr.r0);
  reinterpret_cast<uint4 *>(&tbl[0][0])[lane] = make_uint4(0, 0, 0, 0);
  wave_sync();
  // sort key of entry `lane` of run d: offset in its bucket (< 2^20) << 31 | index
  const uint64_t offmask = (uint64_t(1) << lgt) - 1;
  uint64_t key[SL];
  uint32_t head = CMIN_NONE;
#pragma unroll
  for (int d = 0; d < SL; d++) {
    const uint32_t lend = __builtin_amdgcn_readlane(len, d);
    const uint64_t rel = xv[d] >> 32;
    key[d] = KEY_ONE | (rel & offmask) << 31 | (xv[d] & 0xFFFFFFFFull);
    if (d < R && lane < lend) tbl[rel >> lgt][d] = (uint8_t)(lane + 1);
    // a run's first entry has its smallest index (die order is index order)
    const uint32_t ix0 = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)xv[d], 0);
    if (d < R && lend > 0) head = min(head, ix0);
  }
  M.head = head;
  wave_sync();
  {
    const uint4 row = reinterpret_cast<const uint4 *>(&tbl[0][0])[lane];
    const uint32_t rw[4] = {row.x, row.y, row.z, row.w};
#pragma unroll
    for (int d = 0; d < SL; d++) {
      const uint32_t y = (rw[d >> 2] >> (8 * (d & 3))) & 0xFFu;
      const uint64_t v = __shfl(key[d], y ? (int)(y - 1) : 0);
      M.slot[d] = y ? v : KEY_EMPTY;
      M.cnt += y ? 1u : 0u;
    }
  }
  sort_slots<SL>(M.slot);
  M.boff = wave_excl_sum(M.cnt);
  const int64_t cst = cstart + ((int64_t)lane << lgt) - M.rank0 * xfer;
#pragma unroll
  for (int i = 0; i < SL; i++) {
    if ((uint32_t)i < M.cnt) {
      const int64_t v = cst + (int64_t)((M.slot[i] >> 31) & 0x1FFFFFu) - (int64_t)mul32(M.boff + i, (uint32_t)xfer);
      M.loc = imax(M.loc, v);
    }
  }
  wave_sync();  // tbl is reused by the wave's next cell
}

// Completions of a merged cell given its entering term gin: staged in the
// band when they fit, else stored directly.  mytop: staged span used.
template <int SL>
DEVI void cell_emit(const Merged<SL> &M, const Geo &g, int64_t cstart, int64_t gin, uint32_t lo, int64_t wbase,
                    uint32_t *stage, int64_t *__restrict__ complete, uint32_t n, uint32_t *errb,
                    uint32_t &mytop) {
  if (M.m == 0) return;
  const uint32_t lane = lane_id();
  const int64_t xfer = g.xfer;
  const int64_t cst = cstart + ((int64_t)lane << g.lg_tR) - M.rank0 * xfer;
  int64_t carry = __shfl_up(wave_incl_max(M.loc), 1);
  if (lane == 0) carry = NEG;
  carry = imax(carry, gin);
  const int64_t r0x = M.rank0 * xfer;
#pragma unroll
  for (int i = 0; i < SL; i++) {
    if ((uint32_t)i < M.cnt) {
      const int64_t v = cst + (int64_t)((M.slot[i] >> 31) & 0x1FFFFFu) - (int64_t)mul32(M.boff + i, (uint32_t)xfer);
      carry = imax(carry, v);
      const int64_t cpl = r0x + (int64_t)mul32(M.boff + i + 1, (uint32_t)xfer) + carry;
      if (cpl >= TIME_LIMIT) *errb |= ERR_OVERFLOW;
      const uint32_t ix = (uint32_t)M.slot[i] & 0x7FFFFFFFu;
      if (ix < n) {
        const uint32_t rel = ix - lo;
        const uint64_t off = (uint64_t)(cpl - wbase);
        if (ix >= lo && rel < WIN_SLOTS && off < WIN_EMPTY) {
          stage[win_slot(rel)] = (uint32_t)off;
          mytop = max(mytop, rel + 1);
        } else {
          complete[ix] = cpl;
        }
      }
    }
  }
}

// Requests of channel c in the call (lanes < Dk read one die queue each).
DEVI uint32_t chan_total(const uint32_t *__restrict__ totals, uint32_t Dk, uint32_t c) {
  const uint32_t lane = lane_id();
  return wave_sum(lane < Dk ? totals[c * Dk + lane] : 0u);
}

template <int SL>
__global__ __launch_bounds__(WIN_THREADS) void k_cell_chan(
    const int64_t *__restrict__ DD, const uint32_t *__restrict__ LB, const uint32_t *__restrict__ seg_start,
    const uint32_t *__restrict__ totals, Geo g, CallCtl *ctl, const DevState *st, uint64_t *WAGG, uint64_t *WINC,
    int64_t *__restrict__ complete, int64_t *__restrict__ cfnew, uint32_t gmax, uint32_t n) {
  extern __shared__ __align__(16) unsigned char smem[];
  WinLds &S = *(WinLds *)smem;
  if (agent_load32(&ctl->err)) return;
  const uint32_t G = ctl->G, shift = ctl->shift, C = g.C;
  if (G == 0 || !grid_bucketable<SL>(g, shift)) return;
  const int64_t cbase = ctl->cbase, xfer = g.xfer;
  const uint32_t t = threadIdx.x, w = t >> 6, lane = t & 63;
  const uint32_t NG = (C + CH_GROUP - 1) / CH_GROUP;
  const uint32_t U = G * NG;
  for (uint32_t q = t; q < WIN_SLOTS; q += WIN_THREADS) S.stage[q] = WIN_EMPTY;
  uint32_t errb = 0;
  while (true) {
    if (t == 0) S.unit = atomicAdd(&ctl->wctr, 1u);
    __syncthreads();
    const uint32_t u = S.unit;
    if (u >= U) break;  // the same for the whole workgroup
    const uint32_t j = u / NG, c0 = (u - j * NG) * CH_GROUP;
    const int64_t cstart = cbase + ((int64_t)j << shift);
    const uint32_t ca = c0 + w, cb = c0 + w + WIN_WAVES;
    Merged<SL> A, B;
    A.m = B.m = 0;
    if (ca < C) {
      const CellRuns cr = cell_runs(LB, seg_start, totals, g.Dk, gmax, ca, j);
      uint64_t xv[SL];
      load_runs<SL>(DD, cr, (int)g.Dk, xv);
      cell_merge<SL>(S.tbl[w], cr, xv, g, cstart, A, &errb);
    }
    if (cb < C) {
      const CellRuns cr = cell_runs(LB, seg_start, totals, g.Dk, gmax, cb, j);
      uint64_t xv[SL];
      load_runs<SL>(DD, cr, (int)g.Dk, xv);
      cell_merge<SL>(S.tbl[w], cr, xv, g, cstart, B, &errb);
    }
    const int64_t ma = A.m ? wave_max(A.loc) : NEG, mb = B.m ? wave_max(B.loc) : NEG;
    if (lane == 0) {
      if (ca < C) agent_store64(&WAGG[(size_t)ca * gmax + j], enc_time(ma));
      if (cb < C) agent_store64(&WAGG[(size_t)cb * gmax + j], enc_time(mb));
    }
    int64_t ga = NEG, gb = NEG;
    look_back2(WAGG, WINC, C, gmax, j, ca, cb, ca < C ? st->chan_free[ca] : NEG, cb < C ? st->chan_free[cb] : NEG,
               ga, gb, &errb);
    const int64_t ia = imax(ga, ma), ib = imax(gb, mb);
    if (lane == 0) {
      if (ca < C) agent_store64(&WINC[(size_t)ca * gmax + j], enc_time(ia));
      if (cb < C) agent_store64(&WINC[(size_t)cb * gmax + j], enc_time(ib));
    }
    if (j == G - 1) {  // the channels' clocks after the call
      const uint32_t ta = ca < C ? chan_total(totals, g.Dk, ca) : 0u;
      const uint32_t tb = cb < C ? chan_total(totals, g.Dk, cb) : 0u;
      if (lane == 0) {
        if (ca < C) {
          cfnew[ca] = (int64_t)ta * xfer + ia;
          if (ta) atomicMax((long long *)&ctl->max_cpl, (long long)((int64_t)ta * xfer + ia));
        }
        if (cb < C) {
          cfnew[cb] = (int64_t)tb * xfer + ib;
          if (tb) atomicMax((long long *)&ctl->max_cpl, (long long)((int64_t)tb * xfer + ib));
        }
      }
    }
    // band start (smallest index of the unit's requests) and completion base
    // (a lower bound of every completion of the unit)
    uint32_t mn = min(A.m ? A.head : CMIN_NONE, B.m ? B.head : CMIN_NONE);
    int64_t bmin = INT64_MAX;
    if (A.m) bmin = imin(bmin, (A.rank0 + 1) * xfer + ga);
    if (B.m) bmin = imin(bmin, (B.rank0 + 1) * xfer + gb);
    if (lane == 0) {
      S.rmin[w] = mn;
      S.rbase[w] = bmin;
    }
    if (t == 0) S.top = 0;
    __syncthreads();
    uint32_t lo = CMIN_NONE;
    int64_t wbase = INT64_MAX;
#pragma unroll
    for (int k = 0; k < WIN_WAVES; k++) {
      lo = min(lo, S.rmin[k]);
      wbase = imin(wbase, S.rbase[k]);
    }
    if (lo != CMIN_NONE) {  // the same for the whole workgroup
      uint32_t top = 0;
      cell_emit<SL>(A, g, cstart, ga, lo, wbase, S.stage, complete, n, &errb, top);
      cell_emit<SL>(B, g, cstart, gb, lo, wbase, S.stage, complete, n, &errb, top);
      top = wave_umax(top);
      if (lane == 0 && top) atomicMax(&S.top, top);
      __syncthreads();
      const uint32_t used = S.top;
      for (uint32_t q = t; q < used; q += WIN_THREADS) {
        const uint32_t sq = win_slot(q);
        const uint32_t v = S.stage[sq];
        if (v != WIN_EMPTY) {
          complete[lo + q] = wbase + (int64_t)v;
          S.stage[sq] = WIN_EMPTY;
        }
      }
    }
    __syncthreads();
  }
  if (errb) atomicOr(&ctl->err, errb);
}

// Grids off the bucket path: every cell k_cell_agg listed, one wave each,
// streamed through the LDS with its entering term from k_cell_scan,
// completions stored directly.
template <int SL>
__global__ __launch_bounds__(64) void k_cell_rest(
    const int64_t *__restrict__ DD, const uint32_t *__restrict__ IX, const uint32_t *__restrict__ LB,
    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ totals, Geo g, CallCtl *ctl,
    const int64_t *__restrict__ GIN, const uint32_t *__restrict__ NBL, int64_t *__restrict__ complete,
    uint32_t gmax, uint32_t n) {
  extern __shared__ __align__(16) unsigned char smem[];
  CellLds &S = *(CellLds *)smem;
  if (agent_load32(&ctl->err)) return;
  const uint32_t nr = agent_load32(&ctl->n_rest);
  const uint32_t shift = ctl->shift;
  const int64_t cbase = ctl->cbase;
  uint32_t errb = 0;
  for (uint32_t i = blockIdx.x; i < nr; i += gridDim.x) {
    const uint32_t id = NBL[i];
    const uint32_t j = id / g.C, c = id - j * g.C;
    const CellRuns cr = cell_runs(LB, seg_start, totals, g.Dk, gmax, c, j);
    uint64_t xv[SL];
    load_runs<SL>(DD, cr, (int)g.Dk, xv);
    cell_pass<SL, true>(S, DD, IX, cr, xv, g, shift, cbase, j, GIN[(size_t)c * gmax + j], complete, n, &errb);
    wave_sync();
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
  for (uint32_t k = threadIdx.x; k < MAX_KEYS; k += blockDim.x) {
    st->die_free[k] = NEG;
    st->ref_pend[k] = 0;  // pending refresh quanta are dropped
    st->ref_head[k] = 0;
  }
  for (uint32_t c = threadIdx.x; c < MAX_CHANNELS; c += blockDim.x) st->chan_free[c] = NEG;
  if (threadIdx.x == 0) {  // the vmem route: idle, no burst
    st->vfree = NEG;
    st->vlast = 0;
    st->vburst = 0;
    st->vhave = 0;
  }
}

// ------------------------------------------------------------------ refresh bookkeeping

// After a call on the refresh path: die queue k's first min(pending, its
// admissions) quanta were claimed.  Success retires them; a failed call
// claims nothing, so their completion cells go back to pending.
__global__ __launch_bounds__(BLK) void k_refresh_commit(const CallCtl *ctl, DevState *st,
                                                        const uint32_t *__restrict__ totals, uint32_t K) {
  const uint32_t err = agent_load32(&ctl->err);
  for (uint32_t k = blockIdx.x * BLK + threadIdx.x; k < K; k += gridDim.x * BLK) {
    const uint32_t R = st->ref_pend[k], used = min(R, totals[k]);
    if (!used) continue;
    if (err) {
      int64_t *const *q = st->ref_slot + st->ref_off[k] + st->ref_head[k];
      for (uint32_t r = 0; r < used; r++) *q[r] = REFRESH_PENDING;
    } else {
      st->ref_head[k] += used;
      st->ref_pend[k] = R - used;
    }
  }
}

// Idle-window drain: each die queue, oldest quantum first, starts the next
// one at max(its clock, t_from) while it ends by t_to.
__global__ __launch_bounds__(BLK) void k_refresh_drain(DevState *st, uint32_t K, int64_t tQ, int64_t t_from,
                                                       int64_t t_to) {
  const uint32_t k = blockIdx.x * BLK + threadIdx.x;
  if (k >= K) return;
  uint32_t R = st->ref_pend[k], h = st->ref_head[k];
  if (!R) return;
  int64_t t = imax(st->die_free[k], t_from);  // NEG (idle since -inf) -> t_from
  int64_t *const *q = st->ref_slot + st->ref_off[k];
  const uint32_t R0 = R;
  while (R && t + tQ <= t_to) {
    t += tQ;
    *q[h++] = t;
    R--;
  }
  if (R != R0) {
    st->die_free[k] = t;
    st->ref_head[k] = h;
    st->ref_pend[k] = R;
  }
}

__global__ __launch_bounds__(BLK) void k_fill(int64_t *__restrict__ p, int64_t n, int64_t v) {
  for (int64_t i = (int64_t)blockIdx.x * BLK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLK) p[i] = v;
}

// ------------------------------------------------------------------ launchers

const char *const kKernelNames[] = {"k_prologue",  "k_die_reduce", "k_tile_scan", "k_key_scan",
                                    "k_die_scatter", "k_cell_chan", "k_cell_agg",  "k_cell_scan",
                                    "k_cell_rest", "k_finalize",  "k_small"};
const int kNumTimedKernels = 11;
constexpr int SMALL_SLOT = 10;  // k_small's timing slot

static size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

// LDS of pass 1: range table | amax[K], cmax[K] i64 | cnt[K] | wcnt[DWAVES][K] u16 | tot[K] u16 |
// refp[K] u32 | tag[DWAVES][K] u32
size_t lds_die_reduce(uint32_t K) {
  return align16(sizeof(LdsRanges)) + K * (8 + 8 + 4) + DWAVES * K * 2 + K * 2 + 4 + K * 4 + DWAVES * K * 4;
}
size_t lds_die_count(uint32_t K) { return align16(sizeof(LdsRanges)) + K * 4; }
static size_t lds_die_scatter_sc(uint32_t K, int SC) {
  const size_t cp = SC == 2 ? chunk_pad<2>() : chunk_pad<1>();
  return cp * 8 + (size_t)K * (sizeof(KeyA) + sizeof(KeyW) + 4 + 4 + (SC == 2 ? 4 : 0)) + cp * 6;
}
constexpr size_t LDS_MAX = 160 * 1024;
// two chunks per step where their LDS fits
static int die_scatter_sc(uint32_t K) { return lds_die_scatter_sc(K, 2) <= LDS_MAX ? 2 : 1; }
size_t lds_die_scatter(uint32_t K) { return lds_die_scatter_sc(K, die_scatter_sc(K)); }

hipError_t launch_time_requests(const Geo &g, const RangeTable &rt, const Layout &Lo, char *ws,
                                DevState *st, const uint64_t *addr, const int64_t *issue,
                                int64_t *complete, hipStream_t s, hipEvent_t *ev, int n_ev,
                                bool refresh) {
  if (g.vmem) return launch_vmem(g, rt, Lo, ws, st, addr, issue, complete, s);
  CallCtl *ctl = (CallCtl *)(ws + Lo.off_ctl);
  if (small_path_ok(g, Lo.n, refresh)) {  // one launch; timed in its own slot
    for (int i = 0; i <= SMALL_SLOT && ev && i < n_ev; i++) hipEventRecord(ev[i], s);
    const hipError_t es = launch_small(g, rt, st, ctl, addr, issue, Lo.n, complete, s);
    for (int i = SMALL_SLOT + 1; ev && i < n_ev; i++) hipEventRecord(ev[i], s);
    return es;
  }
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
  uint32_t *KR = (uint32_t *)(ws + Lo.off_kr);
  uint32_t *LB = (uint32_t *)(ws + Lo.off_lb);
  int64_t *AGG = (int64_t *)(ws + Lo.off_cagg);
  int64_t *GIN = (int64_t *)(ws + Lo.off_cgin);
  uint64_t *WST = (uint64_t *)(ws + Lo.off_wst);
  const bool p2 = g.pow2 != 0;
  int evi = 0;
  auto mark = [&]() {
    if (ev && evi < n_ev) hipEventRecord(ev[evi++], s);
  };
  hipError_t e;
  mark();
  hipLaunchKernelGGL(k_prologue, dim3(1), dim3(64), 0, s, ctl);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  const dim3 key_waves((g.K + WAVES - 1) / WAVES);
  if (refresh) {
    // count pass and per-tile rank bases first (timed with pass 1)
    const size_t lds = lds_die_count(g.K);
    if (p2)
      hipLaunchKernelGGL(k_die_count<true>, dim3(Lo.nt), dim3(DBLK), lds, s, addr, Lo.n, g, rt, Lo.tile_elems,
                         agg_cnt);
    else
      hipLaunchKernelGGL(k_die_count<false>, dim3(Lo.nt), dim3(DBLK), lds, s, addr, Lo.n, g, rt,
                         Lo.tile_elems, agg_cnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_tile_count, key_waves, dim3(BLK), 0, s, agg_cnt, Lo.nt, g.K, tin_base, totals);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    const size_t lds = lds_die_reduce(g.K);
    auto kfn = p2 ? (refresh ? k_die_reduce<true, true> : k_die_reduce<true, false>)
                  : (refresh ? k_die_reduce<false, true> : k_die_reduce<false, false>);
    hipLaunchKernelGGL(kfn, dim3(Lo.nt), dim3(DBLK), lds, s, addr, issue, Lo.n, complete, g, rt, Lo.tile_elems,
                       agg_cnt, agg_A, KR, ctl, tin_base, st);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  if (refresh)
    hipLaunchKernelGGL(k_tile_scan_ref, key_waves, dim3(BLK), 0, s, agg_A, Lo.nt, g, st, tin_base, totals, tin_L,
                       dfnew, ctl);
  else
    hipLaunchKernelGGL(k_tile_scan, key_waves, dim3(BLK), 0, s, agg_cnt, agg_A, Lo.nt, g.K, g.tR, st, tin_L,
                       tin_base, totals, dfnew, ctl);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  hipLaunchKernelGGL(k_key_scan, dim3(1), dim3(BLK), 0, s, totals, g.K, seg, issue, Lo.gmax, Lo.s0, ctl);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  {
    const size_t lds = lds_die_scatter(g.K);
    const bool two = die_scatter_sc(g.K) == 2;
    hipLaunchKernelGGL(refresh ? (two ? k_die_scatter<true, 2> : k_die_scatter<true, 1>)
                               : (two ? k_die_scatter<false, 2> : k_die_scatter<false, 1>),
                       dim3(Lo.nt), dim3(SBLK), lds, s,
                       issue, KR, Lo.n, g, Lo.tile_elems, tin_L, tin_base, seg, totals, DD, IX, LB, Lo.gmax, ctl,
                       st, WST, g.reg_block ? (int64_t *)(ws + Lo.off_iss) : (int64_t *)nullptr);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark();
  if (g.reg_block) {
    // media variant: the channel stage simulated per channel in service
    // order (timed in the first channel-stage slot)
    if ((e = launch_regblock(g, (const uint64_t *)DD, IX, (const int64_t *)(ws + Lo.off_iss), seg, totals, st, ctl,
                             complete, dfnew, cfnew, refresh, s)) != hipSuccess)
      return e;
    mark();
    mark();
    mark();
  } else {
    // channel stage.  On the bucket path (every grid but those with very
    // wide cells or more than 16 die queues per channel) k_cell_chan does
    // all of it; otherwise k_cell_agg -> k_cell_scan -> k_cell_rest.  Each
    // kernel reads the grid the die stage chose and returns at once when
    // the stage is the other one's.
    int dev = 0, ncu = 256, per_cu = 0;
    hipGetDevice(&dev);
    hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    const int sl = g.Dk <= 4 ? 4 : g.Dk <= 8 ? 8 : 16;
    const uint32_t nn = (uint32_t)Lo.n;
    uint64_t *WAGG = WST, *WINC = WST + (size_t)Lo.gmax * g.C;
    {  // one 1,024-thread workgroup per CU (its LDS holds a unit's band)
      const dim3 gw((uint32_t)ncu), bw(WIN_THREADS);
      const size_t lw = sizeof(WinLds);
      if (sl == 4)
        hipLaunchKernelGGL(k_cell_chan<4>, gw, bw, lw, s, DD, LB, seg, totals, g, ctl, st, WAGG, WINC, complete,
                           cfnew, Lo.gmax, nn);
      else if (sl == 8)
        hipLaunchKernelGGL(k_cell_chan<8>, gw, bw, lw, s, DD, LB, seg, totals, g, ctl, st, WAGG, WINC, complete,
                           cfnew, Lo.gmax, nn);
      else
        hipLaunchKernelGGL(k_cell_chan<16>, gw, bw, lw, s, DD, LB, seg, totals, g, ctl, st, WAGG, WINC, complete,
                           cfnew, Lo.gmax, nn);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    mark();
    // off the bucket path: enough one-wave blocks to fill the chip, a
    // multiple of the XCD count, and no more than there can be cells
    const void *kfn = sl == 4 ? (const void *)k_cell_agg<4>
                      : sl == 8 ? (const void *)k_cell_agg<8> : (const void *)k_cell_agg<16>;
    hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kfn, 64, sizeof(CellLds));
    per_cu = per_cu < 1 ? 1 : (per_cu > 32 ? 32 : per_cu);
    const uint64_t cells = (uint64_t)g.C * Lo.gmax;
    auto grid_of = [&](int waves_per_cu) {
      uint64_t blocks = (uint64_t)ncu * (uint64_t)waves_per_cu;
      const uint64_t need = ((cells + NXCD - 1) / NXCD) * NXCD;
      if (blocks > need) blocks = need;
      blocks = (blocks / NXCD) * NXCD;
      if (blocks < NXCD) blocks = NXCD;
      return dim3((uint32_t)blocks);
    };
    const dim3 gr = grid_of(per_cu);
    const dim3 bl(64);
    const size_t lds = sizeof(CellLds);
    uint32_t *NBL = (uint32_t *)(ws + Lo.off_nbl);
    if (sl == 4)
      hipLaunchKernelGGL(k_cell_agg<4>, gr, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, AGG, NBL, Lo.gmax, nn);
    else if (sl == 8)
      hipLaunchKernelGGL(k_cell_agg<8>, gr, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, AGG, NBL, Lo.gmax, nn);
    else
      hipLaunchKernelGGL(k_cell_agg<16>, gr, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, AGG, NBL, Lo.gmax, nn);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    mark();
    hipLaunchKernelGGL(k_cell_scan, dim3(g.C), dim3(BLK), 0, s, AGG, GIN, totals, g, ctl, st, cfnew, Lo.gmax);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    mark();
    {
      const dim3 gx = grid_of(4);
      if (sl == 4)
        hipLaunchKernelGGL(k_cell_rest<4>, gx, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, GIN, NBL, complete,
                           Lo.gmax, nn);
      else if (sl == 8)
        hipLaunchKernelGGL(k_cell_rest<8>, gx, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, GIN, NBL, complete,
                           Lo.gmax, nn);
      else
        hipLaunchKernelGGL(k_cell_rest<16>, gx, bl, lds, s, DD, IX, LB, seg, totals, g, ctl, GIN, NBL, complete,
                           Lo.gmax, nn);
    }
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
  if (refresh) {
    hipLaunchKernelGGL(k_refresh_commit, dim3((g.K + BLK - 1) / BLK), dim3(BLK), 0, s, ctl, st, totals, g.K);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  mark();
  while (ev && evi < n_ev) mark();  // the remaining slots (k_small's) take no time
  return hipSuccess;
}

hipError_t launch_classify(const Geo &g, const RangeTable &rt, DevState *st, const uint64_t *addr,
                           int64_t n, uint64_t *map, hipStream_t s) {
  // a large grid (a few requests per thread) keeps the most loads in flight:
  // measured 4.7 TB/s at 8,192 blocks against 5.5+ at 131,072 for this
  // read-8-write-8 stream
  int64_t blocks = (n + BLK - 1) / BLK;
  if (blocks > 131072) blocks = 131072;
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

// ------------------------------------------------------------------ closed-loop layers

// Issue time of a layer: t_start for the first, else the previous layer's
// done time + compute_ns (an error value stays negative and fails the layer).
DEVI int64_t layer_time(const int64_t *prev_done, int64_t t_start, int64_t compute_ns) {
  return prev_done ? *prev_done + compute_ns : t_start;
}

__global__ __launch_bounds__(BLK) void k_layer_issue(int64_t *__restrict__ issue, int64_t count,
                                                     const int64_t *prev_done, int64_t t_start,
                                                     int64_t compute_ns) {
  const int64_t t = layer_time(prev_done, t_start, compute_ns);
  for (int64_t i = (int64_t)blockIdx.x * BLK + threadIdx.x; i < count; i += (int64_t)gridDim.x * BLK)
    issue[i] = t;
}

// done = max(t, every completion of the layer), or HBF_TIME_ERROR if the
// layer failed.  Its in-range completions end no later than the last one
// of each channel, which the channel scan recorded in the call's control
// block; native requests complete at t.
__global__ void k_layer_done(const CallCtl *ctl, int64_t count, const int64_t *prev_done, int64_t t_start,
                             int64_t compute_ns, int64_t *done) {
  if (threadIdx.x != 0) return;
  const int64_t t = layer_time(prev_done, t_start, compute_ns);
  int64_t d;
  if (t < 0)
    d = HBF_TIME_ERROR;
  else if (count == 0)
    d = t;
  else if (agent_load32(&ctl->err))
    d = HBF_TIME_ERROR;
  else
    d = imax(t, ctl->max_cpl);
  *done = d;
}

hipError_t launch_layer_issue(int64_t *issue, int64_t count, const int64_t *prev_done, int64_t t_start,
                              int64_t compute_ns, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + BLK - 1) / BLK;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_layer_issue, dim3((uint32_t)blocks), dim3(BLK), 0, s, issue, count, prev_done, t_start,
                     compute_ns);
  return hipGetLastError();
}

hipError_t launch_layer_done(const CallCtl *ctl, int64_t count, const int64_t *prev_done, int64_t t_start,
                             int64_t compute_ns, int64_t *done, hipStream_t s) {
  hipLaunchKernelGGL(k_layer_done, dim3(1), dim3(64), 0, s, ctl, count, prev_done, t_start, compute_ns, done);
  return hipGetLastError();
}

hipError_t set_lds_limits(uint32_t K) {
  hipError_t e;
  const int a = (int)lds_die_reduce(K), b = (int)lds_die_scatter(K), c = (int)lds_die_count(K);
  const void *fa[] = {(const void *)k_die_reduce<true, false>, (const void *)k_die_reduce<false, false>,
                      (const void *)k_die_reduce<true, true>, (const void *)k_die_reduce<false, true>};
  for (const void *f : fa)
    if ((e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, a)) != hipSuccess) return e;
  const void *fb[] = {(const void *)k_die_scatter<false, 1>, (const void *)k_die_scatter<true, 1>,
                      (const void *)k_die_scatter<false, 2>, (const void *)k_die_scatter<true, 2>};
  for (const void *f : fb)
    if ((e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, b)) != hipSuccess) return e;
  const void *fc[] = {(const void *)k_die_count<true>, (const void *)k_die_count<false>};
  for (const void *f : fc)
    if ((e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, c)) != hipSuccess) return e;
  if ((e = set_lds_small()) != hipSuccess) return e;
  const void *fw[] = {(const void *)k_cell_chan<4>, (const void *)k_cell_chan<8>, (const void *)k_cell_chan<16>};
  for (const void *f : fw)
    if ((e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(WinLds))) != hipSuccess)
      return e;
  return hipSuccess;
}

hipError_t launch_refresh_drain(const Geo &g, DevState *st, int64_t t_from, int64_t t_to, hipStream_t s) {
  hipLaunchKernelGGL(k_refresh_drain, dim3((g.K + BLK - 1) / BLK), dim3(BLK), 0, s, st, g.K, g.tQ, t_from, t_to);
  return hipGetLastError();
}

// ------------------------------------------------------------------ static scratch

// Scratch of hbf_time_requests_noalloc: one array per GPU, held until the
// process ends.  In host code `scratch` names a host-side stand-in, not a
// device address; the device address comes from hipGetSymbolAddress, once
// per device, with that device current.
static __device__ __align__(256) char scratch[HBF_NOALLOC_SCRATCH_BYTES];
constexpr int SCRATCH_DEVICES = 64;

hipError_t noalloc_scratch(int dev, char **ptr) {
  static std::mutex mu;
  static char *addr[SCRATCH_DEVICES] = {};
  if (dev < 0 || dev >= SCRATCH_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (uintptr_t)p % 256) return hipErrorInvalidValue;
    addr[dev] = (char *)p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_fill(int64_t *p, int64_t n, int64_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + BLK - 1) / BLK;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill, dim3((uint32_t)blocks), dim3(BLK), 0, s, p, n, v);
  return hipGetLastError();
}

}  // namespace hbf
