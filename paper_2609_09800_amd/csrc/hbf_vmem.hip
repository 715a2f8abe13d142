// The calibrated end-to-end vmem curve as a timing source (HBFSim, arXiv
// 2609.09800, Section "Discussion").  The curve prices a sequential burst of
// L pages, T(L), from knots at 1, 4, 16, 64, 256 and 512 pages (linear in
// between, rounded down to whole ns; beyond 512 the final segment's slope
// continues).  An access extends the current burst only if it reads the
// device page right after the previous in-range access's page; any other
// access starts a one-page burst.  The route serves in-range requests one at
// a time in request order, the access at burst position L taking
// T(L) - T(L-1):
//
//     complete_i = max(issue_i, complete_prev) + c_i
//
// which is a max-plus scan with elements (issue_i + c_i, c_i).  Burst
// positions are a segmented count whose segments break wherever a page does
// not follow its predecessor.  Both are exact integer scans, done in tiles
// of VM_TILE requests:
//
//   k_vm_sum    per tile: the burst summary of its in-range requests
//               (first/last page, count, first and last segment lengths);
//   k_vm_scan1  one block: summaries before each tile (seeded with the
//               route's state from earlier calls);
//   k_vm_cost   per tile: each request's burst position and service
//               (stored), issue-time validation, the tile's max-plus pair;
//   k_vm_scan2  one block: the route clock entering each tile;
//   k_vm_out    per tile: complete[] in request order;
//   k_vm_end    fail-closed fill on error, else commit the route state.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_device.h"
#include "hbf_internal.h"

namespace hbf {

constexpr int VM_WAVES = VM_THREADS / 64;
constexpr uint32_t VM_NATIVE = 0xFFFFFFFFu;  // service slot of a native-path request

// Burst summary of a run of requests (in-range ones only; n = 0: none).
struct VSum {
  uint64_t fp, lp;    // first and last device page
  uint32_t n;         // in-range requests
  uint32_t lead;      // length of the first burst segment
  uint32_t tail;      // length of the last burst segment
  uint32_t whole;     // 1: one segment throughout
};

DEVI VSum vs_none() { return VSum{0, 0, 0, 0, 0, 0}; }
DEVI VSum vs_one(uint64_t page) { return VSum{page, page, 1, 1, 1, 1}; }

// a then b
DEVI VSum vs_comb(const VSum &a, const VSum &b) {
  if (a.n == 0) return b;
  if (b.n == 0) return a;
  const bool join = b.fp == a.lp + 1;
  VSum r;
  r.fp = a.fp;
  r.lp = b.lp;
  r.n = a.n + b.n;
  r.whole = (a.whole && b.whole && join) ? 1u : 0u;
  r.lead = a.whole ? (join ? a.n + b.lead : a.n) : a.lead;
  r.tail = b.whole ? (join ? a.tail + b.n : b.n) : b.tail;
  return r;
}

DEVI VSum vs_shfl_up(const VSum &v, int d) {
  VSum r;
  r.fp = __shfl_up(v.fp, d);
  r.lp = __shfl_up(v.lp, d);
  r.n = __shfl_up(v.n, d);
  r.lead = __shfl_up(v.lead, d);
  r.tail = __shfl_up(v.tail, d);
  r.whole = __shfl_up(v.whole, d);
  return r;
}

// Inclusive scans over the 64 lanes of a wave, in lane order (lane order is
// request order within a round of 64 consecutive requests), on DPP lane
// moves (row shifts by 1, 2, 4, 8, then row broadcasts), lanes without a
// source taking the identity.
template <int CTRL, int ROWMASK>
DEVI uint64_t dpp_u64(uint64_t x) {
  return ((uint64_t)dpp32<CTRL, ROWMASK>(0u, (uint32_t)(x >> 32)) << 32) | dpp32<CTRL, ROWMASK>(0u, (uint32_t)x);
}
template <int CTRL, int ROWMASK>
DEVI VSum vs_dpp(const VSum &x) {
  VSum y;
  y.fp = dpp_u64<CTRL, ROWMASK>(x.fp);
  y.lp = dpp_u64<CTRL, ROWMASK>(x.lp);
  y.n = dpp32<CTRL, ROWMASK>(0u, x.n);
  y.lead = dpp32<CTRL, ROWMASK>(0u, x.lead);
  y.tail = dpp32<CTRL, ROWMASK>(0u, x.tail);
  y.whole = dpp32<CTRL, ROWMASK>(0u, x.whole);
  return y;
}
DEVI VSum vs_wave_incl(VSum x) {
  x = vs_comb(vs_dpp<DPP_ROW_SHR1, 0xF>(x), x);
  x = vs_comb(vs_dpp<DPP_ROW_SHR2, 0xF>(x), x);
  x = vs_comb(vs_dpp<DPP_ROW_SHR4, 0xF>(x), x);
  x = vs_comb(vs_dpp<DPP_ROW_SHR8, 0xF>(x), x);
  x = vs_comb(vs_dpp<DPP_ROW_BCAST15, 0xA>(x), x);
  x = vs_comb(vs_dpp<DPP_ROW_BCAST31, 0xC>(x), x);
  return x;
}

DEVI uint64_t readlane_u64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
}
DEVI uint32_t readlane_u32(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }

// lane l's value, in every lane
DEVI VSum vs_lane(const VSum &v, int l) {
  VSum r;
  r.fp = readlane_u64(v.fp, l);
  r.lp = readlane_u64(v.lp, l);
  r.n = readlane_u32(v.n, l);
  r.lead = readlane_u32(v.lead, l);
  r.tail = readlane_u32(v.tail, l);
  r.whole = readlane_u32(v.whole, l);
  return r;
}

// Max-plus pair: applied to a route clock f it gives max(a, f + b).
struct MP {
  int64_t a, b;
};
DEVI MP mp_none() { return MP{NEG, 0}; }
DEVI MP mp_comb(const MP &x, const MP &y) { return MP{imax(y.a, x.a + y.b), x.b + y.b}; }
DEVI int64_t mp_apply(const MP &p, int64_t f) { return imax(p.a, f + p.b); }

template <int CTRL, int ROWMASK>
DEVI MP mp_dpp(const MP &x) {
  return MP{dpp64<CTRL, ROWMASK>(NEG, x.a), dpp64<CTRL, ROWMASK>(0, x.b)};
}
DEVI MP mp_wave_incl(MP x) {
  x = mp_comb(mp_dpp<DPP_ROW_SHR1, 0xF>(x), x);
  x = mp_comb(mp_dpp<DPP_ROW_SHR2, 0xF>(x), x);
  x = mp_comb(mp_dpp<DPP_ROW_SHR4, 0xF>(x), x);
  x = mp_comb(mp_dpp<DPP_ROW_SHR8, 0xF>(x), x);
  x = mp_comb(mp_dpp<DPP_ROW_BCAST15, 0xA>(x), x);
  x = mp_comb(mp_dpp<DPP_ROW_BCAST31, 0xC>(x), x);
  return x;
}

DEVI MP mp_lane(const MP &v, int l) {
  return MP{(int64_t)readlane_u64((uint64_t)v.a, l), (int64_t)readlane_u64((uint64_t)v.b, l)};
}

// Tile layout: wave w of the tile's workgroup owns requests
// [w * VM_WAVE_SPAN, (w + 1) * VM_WAVE_SPAN) of it, in VM_ITEMS rounds of 64
// consecutive requests (lane = position in the round): every load and store
// instruction touches 64 consecutive elements.
constexpr int64_t VM_WAVE_SPAN = 64 * VM_ITEMS;

// T(L): cost of a sequential burst of L pages.  Knots are nondecreasing
// with at most 2^29 ns per page, so every product below fits int64.
DEVI int64_t vm_burst(const Geo &g, int64_t L) {
  if (L <= 0) return 0;
  const int64_t *T = g.vknot;
  if (L > 512) {
    // floor(d * m / 256) with d = 256 q + r: q m + floor(r m / 256)
    const int64_t d = T[5] - T[4], m = L - 512;
    return T[5] + (d >> 8) * m + (((d & 255) * m) >> 8);
  }
  // the segment [knot s, knot s + 1] holding L; the divisors are constants
  // (segment lengths 3, 12, 48, 192, 256 pages) so that no general 64-bit
  // division is emitted
  const uint64_t u = (uint64_t)L;
  if (u <= 4) return T[0] + (int64_t)((uint64_t)(T[1] - T[0]) * (u - 1) / 3u);
  if (u <= 16) return T[1] + (int64_t)((uint64_t)(T[2] - T[1]) * (u - 4) / 12u);
  if (u <= 64) return T[2] + (int64_t)((uint64_t)(T[3] - T[2]) * (u - 16) / 48u);
  if (u <= 256) return T[3] + (int64_t)((uint64_t)(T[4] - T[3]) * (u - 64) / 192u);
  return T[4] + (int64_t)((uint64_t)(T[5] - T[4]) * (u - 256) >> 8);
}

DEVI uint32_t vm_cost(const Geo &g, int64_t L) { return (uint32_t)(vm_burst(g, L) - vm_burst(g, L - 1)); }

// Device page of an in-range address, or VM_NONE.
constexpr uint64_t VM_NONE = ~uint64_t(0);
DEVI uint64_t vm_page(const Geo &g, const LdsRanges *lr, uint64_t a) {
  const int r = find_range(lr, a);
  if (r < 0) return VM_NONE;
  return g.pow2 ? dev_page<true>(g, lr, r, a) : dev_page<false>(g, lr, r, a);
}

// ------------------------------------------------------------------ kernels

__global__ __launch_bounds__(VM_THREADS) void k_vm_sum(const uint64_t *__restrict__ addr, int64_t n, Geo g,
                                                       RangeTable rt, VSum *__restrict__ TS,
                                                       VSum *__restrict__ WS) {
  __shared__ LdsRanges lr;
  __shared__ VSum sh[VM_WAVES];
  load_ranges(&lr, rt);
  __syncthreads();
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t i0 = (int64_t)blockIdx.x * VM_TILE + w * VM_WAVE_SPAN + lane;
  VSum carry = vs_none();
#pragma unroll 4
  for (int e = 0; e < VM_ITEMS; e++) {
    const int64_t i = i0 + e * 64;
    VSum v = vs_none();
    if (i < n) {
      const uint64_t p = vm_page(g, &lr, addr[i]);
      if (p != VM_NONE) v = vs_one(p);
    }
    carry = vs_comb(carry, vs_lane(vs_wave_incl(v), 63));
  }
  if (lane == 0) {
    sh[w] = carry;
    WS[(size_t)blockIdx.x * VM_WAVES + w] = carry;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    VSum t = vs_none();
    for (int k = 0; k < VM_WAVES; k++) t = vs_comb(t, sh[k]);
    TS[blockIdx.x] = t;
  }
}

// The summary before each tile: one block; thread t folds a contiguous
// group of tiles, a block scan composes the groups, and each thread walks
// its group again.  Seeded with the route's state from earlier calls.
__global__ __launch_bounds__(1024) void k_vm_scan1(const VSum *__restrict__ TS, uint32_t nt,
                                                   VSum *__restrict__ TIN, const DevState *st,
                                                   VSum *__restrict__ vend) {
  __shared__ VSum sh[16];
  const uint32_t per = (nt + 1023) / 1024;
  const uint32_t a = min(nt, threadIdx.x * per), b = min(nt, a + per);
  VSum v = vs_none();
  for (uint32_t t = a; t < b; t++) v = vs_comb(v, TS[t]);
  // the state from earlier calls: a burst of st->vburst pages ending at st->vlast
  VSum seed = vs_none();
  if (st->vhave) {
    seed.fp = seed.lp = st->vlast;
    seed.n = 1;
    seed.lead = seed.tail = (uint32_t)st->vburst;
    seed.whole = 0;
  }
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const VSum x = vs_wave_incl(v);
  if (lane == 63) sh[w] = x;
  __syncthreads();
  VSum before = seed;
  for (int k = 0; k < w; k++) before = vs_comb(before, sh[k]);
  VSum ex = vs_shfl_up(x, 1);
  ex = lane == 0 ? before : vs_comb(before, ex);
  VSum run = ex;
  for (uint32_t t = a; t < b; t++) {
    TIN[t] = run;
    run = vs_comb(run, TS[t]);
  }
  if (threadIdx.x == 1023) *vend = run;
}

// Per tile: burst positions, services (stored for the output pass), issue
// validation, and the max-plus pair of each wave's span and of the tile.
// A wave's entering summary is the tile's prefix and the spans of the
// tile's earlier waves (from k_vm_sum).
__global__ __launch_bounds__(VM_THREADS) void k_vm_cost(const uint64_t *__restrict__ addr,
                                                        const int64_t *__restrict__ issue, int64_t n, Geo g,
                                                        RangeTable rt, const VSum *__restrict__ TIN,
                                                        const VSum *__restrict__ WS, uint32_t *__restrict__ cost,
                                                        MP *__restrict__ TP, MP *__restrict__ WP, CallCtl *ctl) {
  __shared__ LdsRanges lr;
  __shared__ MP shm[VM_WAVES];
  load_ranges(&lr, rt);
  __syncthreads();
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t i0 = (int64_t)blockIdx.x * VM_TILE + w * VM_WAVE_SPAN + lane;
  VSum carry = TIN[blockIdx.x];
  for (int k = 0; k < w; k++) carry = vs_comb(carry, WS[(size_t)blockIdx.x * VM_WAVES + k]);
  uint32_t errb = 0;
  int64_t prev_last = 0;  // issue time of the request before this round's first
  if (lane == 0 && i0 > 0 && i0 - 1 < n) prev_last = issue[i0 - 1];
  MP pair = mp_none();
#pragma unroll 4
  for (int e = 0; e < VM_ITEMS; e++) {
    const int64_t i = i0 + e * 64;
    uint64_t p = VM_NONE;
    int64_t x = 0;
    if (i < n) {
      p = vm_page(g, &lr, addr[i]);
      x = issue[i];
      if (x < 0 || x >= ISSUE_LIMIT) errb |= ERR_RANGE_TIME;
    }
    int64_t before = __shfl_up(x, 1);
    if (lane == 0) before = prev_last;
    if (i < n && i > 0 && x < before) errb |= ERR_UNSORTED;
    prev_last = (int64_t)readlane_u64((uint64_t)x, 63);
    const bool in = p != VM_NONE;
    const VSum inc = vs_wave_incl(in ? vs_one(p) : vs_none());
    // with this request included, the last segment's length is its burst position
    const VSum full = vs_comb(carry, inc);
    MP el = mp_none();
    if (i < n) {
      uint32_t c = VM_NATIVE;
      if (in) {
        c = vm_cost(g, (int64_t)full.tail);
        el = MP{x + (int64_t)c, (int64_t)c};
      }
      cost[i] = c;
    }
    pair = mp_comb(pair, mp_lane(mp_wave_incl(el), 63));
    carry = vs_comb(carry, vs_lane(inc, 63));
  }
  if (lane == 0) {
    shm[w] = pair;
    WP[(size_t)blockIdx.x * VM_WAVES + w] = pair;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    MP t = mp_none();
    for (int k = 0; k < VM_WAVES; k++) t = mp_comb(t, shm[k]);
    TP[blockIdx.x] = t;
  }
  if (errb) atomicOr(&ctl->err, errb);
}

// The route clock entering each tile (one block, as k_vm_scan1), the
// clock after the call, and its largest in-range completion (the last one:
// the route serves in order).
__global__ __launch_bounds__(1024) void k_vm_scan2(const MP *__restrict__ TP, uint32_t nt, int64_t *__restrict__ FIN,
                                                   const DevState *st, CallCtl *ctl, int64_t *__restrict__ vclock) {
  __shared__ MP sh[16];
  if (agent_load32(&ctl->err)) return;
  const uint32_t per = (nt + 1023) / 1024;
  const uint32_t a = min(nt, threadIdx.x * per), b = min(nt, a + per);
  MP v = mp_none();
  for (uint32_t t = a; t < b; t++) v = mp_comb(v, TP[t]);
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const MP x = mp_wave_incl(v);
  if (lane == 63) sh[w] = x;
  __syncthreads();
  MP before = mp_none();
  for (int k = 0; k < w; k++) before = mp_comb(before, sh[k]);
  MP ex;
  ex.a = __shfl_up(x.a, 1);
  ex.b = __shfl_up(x.b, 1);
  ex = lane == 0 ? before : mp_comb(before, ex);
  const int64_t f0 = st->vfree;  // NEG when idle
  int64_t f = mp_apply(ex, f0);
  for (uint32_t t = a; t < b; t++) {
    FIN[t] = f;
    f = mp_apply(TP[t], f);
  }
  if (threadIdx.x == 1023) {
    // everything: a pair whose first term is above NEG holds an in-range request
    const MP all = mp_comb(ex, v);
    *vclock = f;
    ctl->max_cpl = all.a > NEG / 2 ? f : NEG;
    if (f >= TIME_LIMIT) atomicOr(&ctl->err, ERR_OVERFLOW);
  }
}

// complete[] per tile: a wave's entering clock is the tile's, advanced over
// the spans of the tile's earlier waves (pairs from k_vm_cost).
__global__ __launch_bounds__(VM_THREADS) void k_vm_out(const int64_t *__restrict__ issue, int64_t n,
                                                       const uint32_t *__restrict__ cost,
                                                       const int64_t *__restrict__ FIN,
                                                       const MP *__restrict__ WP, int64_t *__restrict__ complete,
                                                       CallCtl *ctl) {
  if (agent_load32(&ctl->err)) return;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int64_t i0 = (int64_t)blockIdx.x * VM_TILE + w * VM_WAVE_SPAN + lane;
  int64_t f = FIN[blockIdx.x];
  for (int k = 0; k < w; k++) f = mp_apply(WP[(size_t)blockIdx.x * VM_WAVES + k], f);
  uint32_t errb = 0;
#pragma unroll 4
  for (int e = 0; e < VM_ITEMS; e++) {
    const int64_t i = i0 + e * 64;
    int64_t x = 0;
    uint32_t c = VM_NATIVE;
    if (i < n) {
      x = issue[i];
      c = cost[i];
    }
    const bool in = c != VM_NATIVE;
    const MP inc = mp_wave_incl(in ? MP{x + (int64_t)c, (int64_t)c} : mp_none());
    if (i < n) {
      if (!in) {
        complete[i] = x;  // native path: no modeled delay
      } else {
        const int64_t t = mp_apply(inc, f);  // this request's completion
        if (t >= TIME_LIMIT) errb |= ERR_OVERFLOW;
        complete[i] = t;
      }
    }
    f = mp_apply(mp_lane(inc, 63), f);
  }
  if (errb) atomicOr(&ctl->err, errb);
}

__global__ __launch_bounds__(256) void k_vm_end(int64_t *__restrict__ complete, int64_t n, CallCtl *ctl,
                                                DevState *st, const VSum *vend, const int64_t *vclock) {
  const uint32_t err = agent_load32(&ctl->err);
  if (err) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
      complete[i] = HBF_TIME_ERROR;
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&st->sticky, err);
    return;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const VSum e = *vend;
    if (e.n) {
      st->vfree = *vclock;
      st->vlast = e.lp;
      st->vburst = e.tail;
      st->vhave = 1;
    }
  }
}

// Prologue of a vmem call: the per-call control block.
__global__ void k_vm_prologue(CallCtl *ctl) {
  if (threadIdx.x == 0) {
    ctl->err = 0;
    ctl->n_in = 0;
    ctl->G = 0;
    ctl->shift = 0;
    ctl->max_dd = NEG;
    ctl->max_cpl = NEG;
    ctl->cbase = 0;
    ctl->n_rest = 0;
  }
}

hipError_t launch_vmem(const Geo &g, const RangeTable &rt, const Layout &L, char *ws, DevState *st,
                       const uint64_t *addr, const int64_t *issue, int64_t *complete, hipStream_t s) {
  CallCtl *ctl = (CallCtl *)(ws + L.off_ctl);
  VSum *TS = (VSum *)(ws + L.off_vsum);
  VSum *TIN = (VSum *)(ws + L.off_vin);
  MP *TP = (MP *)(ws + L.off_vpair);
  int64_t *FIN = (int64_t *)(ws + L.off_vfin);
  uint32_t *cost = (uint32_t *)(ws + L.off_vcost);
  VSum *vend = (VSum *)(ws + L.off_vend);
  VSum *WS = (VSum *)(ws + L.off_vwsum);
  MP *WP = (MP *)(ws + L.off_vwpair);
  int64_t *vclock = (int64_t *)(vend + 1);
  const int64_t n = L.n;
  const uint32_t nt = (uint32_t)((n + VM_TILE - 1) / VM_TILE);
  hipLaunchKernelGGL(k_vm_prologue, dim3(1), dim3(64), 0, s, ctl);
  hipLaunchKernelGGL(k_vm_sum, dim3(nt), dim3(VM_THREADS), 0, s, addr, n, g, rt, TS, WS);
  hipLaunchKernelGGL(k_vm_scan1, dim3(1), dim3(1024), 0, s, TS, nt, TIN, st, vend);
  hipLaunchKernelGGL(k_vm_cost, dim3(nt), dim3(VM_THREADS), 0, s, addr, issue, n, g, rt, TIN, WS, cost, TP, WP,
                     ctl);
  hipLaunchKernelGGL(k_vm_scan2, dim3(1), dim3(1024), 0, s, TP, nt, FIN, st, ctl, vclock);
  hipLaunchKernelGGL(k_vm_out, dim3(nt), dim3(VM_THREADS), 0, s, issue, n, cost, FIN, WP, complete, ctl);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_vm_end, dim3((uint32_t)blocks), dim3(256), 0, s, complete, n, ctl, st, vend, vclock);
  return hipGetLastError();
}

}  // namespace hbf
