// Device-side helpers shared by the HIP kernel files: integer utilities,
// wave64 cross-lane scans (DPP), block scans, and classification of an
// address against the LDS copy of the registered-range snapshot.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

#define DEVI __device__ __forceinline__

DEVI int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }
DEVI int64_t imin(int64_t a, int64_t b) { return a < b ? a : b; }

DEVI uint32_t lane_id() { return __lane_id(); }

// 32 x 32 -> 64-bit product (one v_mad_u64_u32)
DEVI uint64_t mul32(uint32_t a, uint32_t b) { return (uint64_t)a * (uint64_t)b; }

// LDS index padding of the die-order staging arrays: one slot per 16
// (measured: fewer bank conflicts than one per 8 for the blocked scan).
DEVI uint32_t pad16(uint32_t p) { return p + (p >> 4); }

// number of lanes below this one whose bit is set in `mask`
DEVI uint32_t mask_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

DEVI uint32_t agent_load32(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// ------------------------------------------------------------------ block scans

// Exclusive prefix sum over a block of NW waves; returns the block total.
template <int NW>
DEVI uint32_t block_excl_sum(uint32_t v, uint32_t *excl, uint32_t *sh /*[NW]*/) {
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
  for (int i = 0; i < NW; i++) {
    uint32_t t = sh[i];
    base += (i < (int)w) ? t : 0u;
    tot += t;
  }
  __syncthreads();
  *excl = base + x - v;
  return tot;
}

// Exclusive prefix max over a block of NW waves; identity NEG.
template <int NW>
DEVI int64_t block_excl_max(int64_t v, int64_t *sh /*[NW]*/) {
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
  for (int i = 0; i < NW; i++)
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
template <int NW>
DEVI SegMax block_excl_segmax(SegMax v, SegMax *sh /*[NW]*/) {
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
  for (int i = 0; i < NW; i++)
    if (i < (int)w) pre = seg_comb(pre, sh[i]);
  __syncthreads();
  return seg_comb(pre, ex);
}

// ------------------------------------------------------------------ wave-level helpers

DEVI void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}
// DPP cross-lane moves (gfx9 row_shr / row_bcast): lanes without a source, or
// in rows outside ROWMASK, keep `old`.
template <int CTRL, int ROWMASK>
DEVI uint32_t dpp32(uint32_t old, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROWMASK, 0xF, false);
}
template <int CTRL, int ROWMASK>
DEVI int64_t dpp64(int64_t old, int64_t x) {
  const uint32_t lo = dpp32<CTRL, ROWMASK>((uint32_t)old, (uint32_t)x);
  const uint32_t hi = dpp32<CTRL, ROWMASK>((uint32_t)((uint64_t)old >> 32), (uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114, DPP_ROW_SHR8 = 0x118;
constexpr int DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;
// whole-wave shift right by one lane (gfx9 DPP wave_shr:1): lane l gets lane l - 1
constexpr int DPP_WAVE_SHR1 = 0x138;
// Inclusive scans over the 64 lanes: within rows of 16 by shifts of 1, 2,
// 4, 8, then row 0 -> 1 and 2 -> 3 (bcast15), then rows 0-1 -> 2-3 (bcast31).
DEVI uint32_t wave_incl_sum(uint32_t x) {
  x += dpp32<DPP_ROW_SHR1, 0xF>(0u, x);
  x += dpp32<DPP_ROW_SHR2, 0xF>(0u, x);
  x += dpp32<DPP_ROW_SHR4, 0xF>(0u, x);
  x += dpp32<DPP_ROW_SHR8, 0xF>(0u, x);
  x += dpp32<DPP_ROW_BCAST15, 0xA>(0u, x);
  x += dpp32<DPP_ROW_BCAST31, 0xC>(0u, x);
  return x;
}
DEVI uint32_t wave_incl_umax(uint32_t x) {
  x = max(x, dpp32<DPP_ROW_SHR1, 0xF>(0u, x));
  x = max(x, dpp32<DPP_ROW_SHR2, 0xF>(0u, x));
  x = max(x, dpp32<DPP_ROW_SHR4, 0xF>(0u, x));
  x = max(x, dpp32<DPP_ROW_SHR8, 0xF>(0u, x));
  x = max(x, dpp32<DPP_ROW_BCAST15, 0xA>(0u, x));
  x = max(x, dpp32<DPP_ROW_BCAST31, 0xC>(0u, x));
  return x;
}
DEVI int64_t wave_incl_max(int64_t x) {
  x = imax(x, dpp64<DPP_ROW_SHR1, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR2, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR4, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_SHR8, 0xF>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_BCAST15, 0xA>(NEG, x));
  x = imax(x, dpp64<DPP_ROW_BCAST31, 0xC>(NEG, x));
  return x;
}
DEVI uint32_t lane63(uint32_t x) { return (uint32_t)__builtin_amdgcn_readlane((int)x, 63); }
DEVI int64_t lane63(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)x >> 32), 63);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
DEVI uint32_t wave_sum(uint32_t x) { return lane63(wave_incl_sum(x)); }
DEVI uint32_t wave_excl_sum(uint32_t v) { return wave_incl_sum(v) - v; }
DEVI int64_t wave_max(int64_t x) { return lane63(wave_incl_max(x)); }
DEVI uint32_t wave_umax(uint32_t x) { return lane63(wave_incl_umax(x)); }

// ------------------------------------------------------------------ die-stage ranks

// Stable rank of each item among this wave's items with the same key, in
// (item, lane) order; wcnt is the wave's private per-key counter row and tag
// its private per-key scratch row.  Every lane writes its lane number into
// tag[key] and reads it back: one write per key survives, so a lane that
// reads another lane's number shares its key.  Only those groups (in a
// stream of consecutive pages, none or a few per item) are resolved, one
// ballot each; every other lane is alone with its key in this item.
DEVI void wave_rank(const uint32_t *key, uint32_t *rank, uint16_t *wcnt, uint32_t *tag) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int e = 0; e < DITEMS; e++) {
    const uint32_t k = key[e];
    const bool valid = k != KEY_NONE;
    if (valid) tag[k] = lane;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t lead = valid ? tag[k] : lane;
    uint32_t below = 0, cnt = 1;
    uint64_t dup = __ballot(lead != lane);
    while (dup) {  // the same on every lane
      const uint32_t g = (uint32_t)__builtin_amdgcn_readlane((int)lead, (int)__builtin_ctzll(dup));
      const uint64_t gm = __ballot(lead == g);  // the group, its surviving writer included
      if (lead == g) {
        below = mask_below(gm);
        cnt = (uint32_t)__popcll(gm);
      }
      dup &= ~gm;
    }
    uint32_t prior = 0;
    if (valid) prior = wcnt[k];
    // all reads of this item happen before the group writers' updates
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (valid && below == 0) wcnt[k] = (uint16_t)(prior + cnt);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    rank[e] = prior + below;
  }
}

// After wave_rank: turn wcnt[w][k] into the wave's exclusive offset among
// the block's waves and write the chunk total of key k to tot[k].
DEVI void cross_wave_offsets(uint16_t *wcnt, uint16_t *tot, uint32_t K) {
  for (uint32_t k = threadIdx.x; k < K; k += DBLK) {
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < DWAVES; w++) {
      uint32_t c = wcnt[w * K + k];
      wcnt[w * K + k] = (uint16_t)run;
      run += c;
    }
    tot[k] = (uint16_t)run;
  }
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

// LDS slot of die queue k in the die passes: die-major, slot = die * C +
// channel (k = channel * Dk + die).  Device pages stripe over the channels
// first, so the die queues of consecutive pages -- the common case inside a
// wave -- sit in consecutive slots instead of Dk apart, which would put a
// wave's per-queue LDS accesses into a few banks.  lkey inverts it.
DEVI uint32_t lslot(const Geo &g, uint32_t k) {
  if (g.pow2) {
    const uint32_t s = (uint32_t)__builtin_ctz(g.Dk);
    return ((k & (g.Dk - 1)) << g.lg_C) | (k >> s);
  }
  const uint32_t c = k / g.Dk;
  return (k - c * g.Dk) * g.C + c;
}
DEVI uint32_t lkey(const Geo &g, uint32_t li) {
  if (g.pow2) {
    const uint32_t s = (uint32_t)__builtin_ctz(g.Dk);
    return ((li & (g.C - 1)) << s) | (li >> g.lg_C);
  }
  const uint32_t d = li / g.C;
  return (li - d * g.C) * g.Dk + d;
}

// The range snapshot's count and its first range, held in registers (read
// once after load_ranges): with a single range the test is one subtraction
// and compare instead of a search through the LDS table.
struct RangeReg {
  int32_t n;
  uint64_t base, bytes, pbase;
};
DEVI RangeReg range_reg(const LdsRanges *lr) {
  return RangeReg{lr->n, lr->base[0], lr->bytes[0], lr->pbase[0]};
}

// Die-queue key of an address, or KEY_NONE for the native path.
template <bool POW2>
DEVI uint32_t key_of(const Geo &g, const LdsRanges *lr, const RangeReg &rr, uint64_t a) {
  uint64_t dp;
  if (rr.n == 1) {
    const uint64_t off = a - rr.base;  // wraps above bytes when a < base
    if (off >= rr.bytes) return KEY_NONE;
    dp = rr.pbase + (POW2 ? (off >> g.lg_page) : off / g.page_bytes);
  } else {
    const int r = find_range(lr, a);
    if (r < 0) return KEY_NONE;
    dp = dev_page<POW2>(g, lr, r, a);
  }
  Loc L = map_page<POW2>(g, dp);
  uint32_t k = L.ch * g.D + L.die;
  if (g.plane_parallel) k = k * g.P + L.plane;
  return k;
}

}  // namespace hbf
