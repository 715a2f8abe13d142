// Closed-loop layered decode (hbf_time_layers), one launch for all layers.
//
// The running program pays each layer's modeled delays before it issues
// the next layer (HBFSim, arXiv 2609.09800, Section "Introduction"; the
// wait sits at first use, Section D2).  Every request of layer l is issued
// at the same time t_l, which makes the two queue stages of the media model
// closed-form within the layer:
//   * die queue k holds m_k of the layer's requests and serves them back to
//     back from base_k = max(t_l, its clock): the j-th (index order) leaves
//     the die at base_k + (j+1)*tR;
//   * a channel serves by (die-done, index), so the channel rank of that
//     request is j plus, for each other die queue k' of the channel, the
//     number of k''s requests that leave their die earlier -- with
//     base_k - base_k' = a*tR + b (floor division), that is a + j + 1 when
//     b > 0 and a + j when b = 0, clamped to [0, m_k'] -- plus one if
//     b = 0 and k''s request a + j (same die-done) has a smaller index;
//   * the channel's completions follow from the Lindley form over that
//     order: complete_r = (r+1)*xfer + max(f0, max_{i<=r} (dd_(i) - i*xfer)).
// Channels only meet through the layer's done time (its latest completion),
// which sets the next layer's issue time.
//
//   k_lay_count  one workgroup per layer: each request's bucket (its die
//                queue, or K for the native path), counts per (layer, bucket)
//   k_lay_scan   one block: bucket offsets, layer-major; clears the
//                per-(layer, channel) done words
//   k_lay_place  one workgroup per layer: each request's index at its
//                bucket's offset + its rank in the bucket (index order)
//   k_lay_run    cooperative, one workgroup per channel, every layer in
//                turn: the channel's completions, then one exchange of
//                the layer's latest completion through the done words.
// The result equals one hbf_time_requests call per layer on the persistent
// model, with the same failure rules: a layer whose issue time is outside
// [0, 2^61) or whose times reach 2^62 fails as a whole (completions
// HBF_TIME_ERROR, clocks untouched, done time HBF_TIME_ERROR), and so does
// every later layer, since its issue time is then negative.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "hbf_device.h"
#include "hbf_internal.h"

namespace hbf {

namespace {

constexpr int LBLK = 512;
constexpr int LWAVES = LBLK / 64;
constexpr int LITEMS = 4;  // completions per thread per scan chunk
constexpr int RBLK = 1024; // k_lay_run: one workgroup per channel
constexpr int RWAVES = RBLK / 64;
constexpr uint32_t LAY_SPIN_ROUNDS = 1u << 24;

// Done words: 0 = not yet published; 1 + error bits for a failed channel
// (< 2^61); else the channel's latest completion + 2^62 (every completion
// and NEG lie in [NEG, 2^62)).
DEVI uint64_t lay_enc(int64_t x) { return (uint64_t)x + (uint64_t(1) << 62); }
DEVI int64_t lay_dec(uint64_t w) { return (int64_t)(w - (uint64_t(1) << 62)); }
constexpr uint64_t LAY_VALID = uint64_t(1) << 61;

// Pre-passes work on tiles of at most LAY_TILE requests of one layer (the
// host lists them: layer, first, end).
struct LayTile {
  int64_t a, b;
  uint32_t layer, first_tile;  // first_tile: the layer's first tile
};

template <bool POW2>
__global__ __launch_bounds__(LBLK) void k_lay_count(const uint64_t *__restrict__ addr, const LayTile *__restrict__ tiles,
                                                    Geo g, RangeTable rt, uint16_t *__restrict__ KEY,
                                                    uint32_t *__restrict__ CNT) {
  extern __shared__ __align__(16) unsigned char smem[];
  LdsRanges *lr = (LdsRanges *)smem;
  uint32_t *cnt = (uint32_t *)(smem + ((sizeof(LdsRanges) + 15) & ~size_t(15)));
  const uint32_t K = g.K;
  const LayTile tl = tiles[blockIdx.x];
  load_ranges(lr, rt);
  for (uint32_t k = threadIdx.x; k <= K; k += LBLK) cnt[k] = 0;
  __syncthreads();
  const RangeReg rr = range_reg(lr);
  for (int64_t i = tl.a + threadIdx.x; i < tl.b; i += LBLK) {
    const uint32_t k0 = key_of<POW2>(g, lr, rr, addr[i]);
    const uint32_t k = k0 == KEY_NONE ? K : k0;
    KEY[i] = (uint16_t)k;
    atomicAdd(&cnt[k], 1u);
  }
  __syncthreads();
  for (uint32_t k = threadIdx.x; k <= K; k += LBLK) CNT[(size_t)blockIdx.x * (K + 1) + k] = cnt[k];
}

// One block per layer: the layer's bucket offsets (from the layer's start;
// OFF[l][K+1] is the layer's end) and each of its tiles' offset in every
// bucket; the layer's done words cleared.
__global__ __launch_bounds__(LBLK) void k_lay_scan(const uint32_t *__restrict__ CNT, const int64_t *__restrict__ ls,
                                                   const uint32_t *__restrict__ tile0, uint32_t K,
                                                   uint32_t *__restrict__ OFF, uint32_t *__restrict__ TOFF,
                                                   uint64_t *__restrict__ SLOT, uint32_t C) {
  __shared__ uint32_t sh[LWAVES];
  const uint32_t l = blockIdx.x, KB = K + 1;
  const uint32_t f = tile0[l], e = tile0[l + 1];
  const uint32_t per = (KB + LBLK - 1) / LBLK;
  const uint32_t k0 = min(KB, threadIdx.x * per), k1 = min(KB, k0 + per);
  uint32_t sum = 0;
  for (uint32_t k = k0; k < k1; k++)
    for (uint32_t q = f; q < e; q++) sum += CNT[(size_t)q * KB + k];
  uint32_t ex;
  block_excl_sum<LWAVES>(sum, &ex, sh);
  uint32_t o = (uint32_t)ls[l] + ex;
  for (uint32_t k = k0; k < k1; k++) {
    OFF[(size_t)l * (KB + 1) + k] = o;
    for (uint32_t q = f; q < e; q++) {
      TOFF[(size_t)q * KB + k] = o;
      o += CNT[(size_t)q * KB + k];
    }
  }
  if (threadIdx.x == 0) OFF[(size_t)l * (KB + 1) + KB] = (uint32_t)ls[l + 1];
  for (uint32_t c = threadIdx.x; c < C; c += LBLK) SLOT[(size_t)l * C + c] = 0;
}

// Each request's index at its tile's offset in its bucket + its rank among
// the tile's requests of that bucket (index order).  Chunks of LBLK
// requests, one per thread: the lanes of a wave that share a bucket are
// found with an LDS tag word (every lane writes its lane number into its
// bucket's word and reads it back; one write survives per bucket), counted
// per wave, and offset by the counts of the chunk's earlier waves and of the
// earlier chunks.
// LDS: run[K+1] u32 | wcnt[LWAVES][K+1] u16 (zero between chunks) | tag[LWAVES][K+1] u32
__global__ __launch_bounds__(LBLK) void k_lay_place(const LayTile *__restrict__ tiles, const uint16_t *__restrict__ KEY,
                                                    uint32_t K, const uint32_t *__restrict__ TOFF,
                                                    uint32_t *__restrict__ LISTD) {
  extern __shared__ __align__(16) unsigned char smem[];
  const uint32_t KB = K + 1;
  uint32_t *run = (uint32_t *)smem;
  uint16_t *wcnt = (uint16_t *)(run + KB);
  uint32_t *tag = (uint32_t *)(((uintptr_t)(wcnt + LWAVES * KB) + 3) & ~(uintptr_t)3);
  for (uint32_t k = threadIdx.x; k < KB; k += LBLK) run[k] = 0;
  for (uint32_t q = threadIdx.x; q < LWAVES * KB; q += LBLK) wcnt[q] = 0;
  __syncthreads();
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  const LayTile tl = tiles[blockIdx.x];
  const uint32_t *off = TOFF + (size_t)blockIdx.x * KB;
  uint32_t *mytag = tag + w * KB;
  for (int64_t c0 = tl.a; c0 < tl.b; c0 += LBLK) {
    const int64_t i = c0 + threadIdx.x;
    const bool valid = i < tl.b;
    const uint32_t k = valid ? KEY[i] : 0u;
    if (valid) mytag[k] = lane;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t lead = valid ? mytag[k] : lane;
    uint32_t below = 0, cnt = 1;
    uint64_t dup = __ballot(lead != lane);
    while (dup) {  // the same on every lane
      const uint32_t gl = (uint32_t)__builtin_amdgcn_readlane((int)lead, (int)__builtin_ctzll(dup));
      const uint64_t gm = __ballot(lead == gl);
      if (lead == gl) {
        below = mask_below(gm);
        cnt = (uint32_t)__popcll(gm);
      }
      dup &= ~gm;
    }
    if (valid && below == 0) wcnt[w * KB + k] = (uint16_t)cnt;
    __syncthreads();
    if (valid) {
      uint32_t r = run[k] + below;
      for (uint32_t v = 0; v < w; v++) r += wcnt[v * KB + k];
      LISTD[off[k] + r] = (uint32_t)i;
    }
    __syncthreads();
    if (valid && below == 0) {
      atomicAdd(&run[k], cnt);
      wcnt[w * KB + k] = 0;
    }
    __syncthreads();
  }
}

DEVI uint32_t wave_or(uint32_t x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x |= (uint32_t)__shfl_xor((int)x, d);
  return x;
}

// Floor division of a by a positive d (int64).
DEVI int64_t floor_div(int64_t a, int64_t d) {
  const int64_t q = a / d;
  return (a % d != 0 && a < 0) ? q - 1 : q;
}

struct LayArgs {
  const int64_t *ls;
  const uint32_t *OFF, *LISTD;
  int64_t *RV;
  uint32_t *RI;
  uint64_t *SLOT;
  int64_t *issue, *complete, *done;
  DevState *st;
  Geo g;
  int64_t t_start, compute_ns;
  uint32_t L;
};

// Channel ranks, Lindley terms and completions of one layer's requests of a
// channel: LI = their request indices by die queue and rank, RV / RI = the
// terms and indices by channel rank.  Inlined twice, on LDS arrays and on
// device-memory arrays, so each copy addresses one memory directly.
template <typename PL, typename PV, typename PI>
DEVI void lay_rank_scan(PL LI, PV RV, PI RI, uint32_t Mc, uint32_t Dk, const uint32_t *boff, const int64_t *base,
                        const uint4 *pairs, int64_t tR, int64_t xfer,
                        int64_t cfree, int64_t *__restrict__ complete, int64_t *shm, int64_t *s_chunk,
                        int64_t *s_last, uint32_t *s_err) {
  const uint32_t t = threadIdx.x;
  // channel rank and Lindley term of each of the channel's requests
  for (uint32_t p = t; p < Mc; p += RBLK) {
    uint32_t lo = 0, hi = Dk;  // the die queue holding entry p: the last d with boff[d] <= p
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (boff[mid] <= p) lo = mid;
      else hi = mid;
    }
    const uint32_t b = lo, j = p - boff[b];
    const uint32_t idx = LI[p];
    const int64_t dd = base[b] + (int64_t)(j + 1) * tR;
    const uint4 *prow = pairs + b * Dk;
    int32_t r = (int32_t)j;
    // branch-free over the other die queues, one 16-byte record each, so
    // their LDS reads overlap; 32-bit throughout (alpha is clamped to +-2^23,
    // beyond any rank)
#pragma unroll 4
    for (uint32_t b1 = 0; b1 < Dk; b1++) {
      const uint4 pr = prow[b1];  // {alpha, beta, m (0 for b itself), first position}
      const int32_t mb = (int32_t)pr.z;
      const int32_t al = (int32_t)pr.x + (int32_t)j;
      const uint32_t be = pr.y;
      const int32_t k0 = min(max(be ? al + 1 : al, 0), mb);  // b1's requests leaving their die earlier
      // the one that leaves at the same time comes first if its index is smaller
      const bool tie = !be && (uint32_t)al < (uint32_t)mb;
      const uint32_t other = LI[tie ? pr.w + (uint32_t)al : p];
      r += k0 + ((tie && other < idx) ? 1 : 0);
    }
    RV[r] = dd - (int64_t)r * xfer;
    RI[r] = idx;
  }
  __syncthreads();
  // Lindley prefix over the channel order, RBLK * LITEMS ranks at a time
  int64_t run = cfree;
  for (uint32_t r0c = 0; r0c < Mc; r0c += RBLK * LITEMS) {
    const uint32_t r0 = r0c + t * LITEMS;
    int64_t v[LITEMS];
    int64_t mx = NEG;
#pragma unroll
    for (int q = 0; q < LITEMS; q++) {
      v[q] = (r0 + q < Mc) ? RV[r0 + q] : NEG;
      mx = imax(mx, v[q]);
    }
    const int64_t ex = block_excl_max<RWAVES>(mx, shm);
    int64_t pre = imax(run, ex);
#pragma unroll
    for (int q = 0; q < LITEMS; q++) {
      if (r0 + q < Mc) {
        pre = imax(pre, v[q]);
        const int64_t cpl = (int64_t)(r0 + q + 1) * xfer + pre;
        if (cpl >= TIME_LIMIT) atomicOr(s_err, ERR_OVERFLOW);
        complete[RI[r0 + q]] = cpl;
        if (r0 + q + 1 == Mc) *s_last = cpl;
      }
    }
    if (t == RBLK - 1) *s_chunk = imax(ex, mx);  // the chunk's maximum
    __syncthreads();
    run = imax(run, *s_chunk);
    __syncthreads();
  }
}

// One workgroup per channel c; every layer in turn.  A layer's requests of
// the channel (at most cap of them) are staged in LDS with their ranks and
// Lindley terms; a larger share of a layer works in the device-memory copies.
// The next layer's offsets and request list are fetched into the other of
// two buffers while wave 0 runs the current layer's exchange.
// LDS: pairs[Dk][Dk] {alpha, beta, m, first position} | dfree[Dk], base[Dk], sRV[cap] i64 |
//      m[Dk], boff[2][Dk+1], sL[2][cap], sRI[cap] u32
struct LayHdr {
  uint32_t oc, Mc, n0, nn, any;
};

__global__ __launch_bounds__(RBLK) void k_lay_run(LayArgs A, uint32_t cap) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int64_t shm[RWAVES];
  __shared__ int64_t s_last, s_chunk, s_lmax;
  __shared__ uint32_t s_err, s_any;
  __shared__ LayHdr hdr[2];
  const Geo &g = A.g;
  const uint32_t Dk = g.Dk, C = g.C, K = g.K, KB = K + 1, c = blockIdx.x;
  const int64_t tR = g.tR, xfer = g.xfer;
  uint4 *pairs = (uint4 *)smem;
  int64_t *dfree = (int64_t *)(pairs + Dk * Dk);
  int64_t *base = dfree + Dk;
  int64_t *sRV = base + Dk;
  uint32_t *m = (uint32_t *)(sRV + cap);
  uint32_t *boffb = m + Dk;  // [2][Dk + 1]
  uint32_t *sLb = boffb + 2 * (Dk + 1);  // [2][cap]
  uint32_t *sRI = sLb + 2 * cap;
  const uint32_t t = threadIdx.x, lane = lane_id();
  // layer ll's offsets and (when it fits) its request list into buffer ll & 1,
  // by threads [t0, RBLK)
  auto fetch = [&](uint32_t ll, uint32_t t0) {
    if (ll >= A.L || t < t0) return;
    const uint32_t u = t - t0, nt = RBLK - t0, bi = ll & 1;
    const uint32_t *off = A.OFF + (size_t)ll * (KB + 1);
    const uint32_t oc = off[c * Dk], Mc = off[(c + 1) * Dk] - oc;
    for (uint32_t d = u; d <= Dk; d += nt) boffb[bi * (Dk + 1) + d] = off[c * Dk + d] - oc;
    if (Mc <= cap)
      for (uint32_t p = u; p < Mc; p += nt) sLb[bi * cap + p] = A.LISTD[oc + p];
    if (u == 0) hdr[bi] = LayHdr{oc, Mc, off[K], off[KB] - off[K], off[KB] > off[0] ? 1u : 0u};
  };
  for (uint32_t d = t; d < Dk; d += RBLK) dfree[d] = A.st->die_free[c * Dk + d];
  int64_t cfree = A.st->chan_free[c];
  int64_t prev_done = 0;
  fetch(0, 0);
  __syncthreads();
  for (uint32_t l = 0; l < A.L; l++) {
    const int64_t tl = l == 0 ? A.t_start : prev_done + A.compute_ns;
    const uint32_t bi = l & 1;
    const LayHdr h = hdr[bi];
    const bool any_req = h.any != 0;  // the layer is not empty
    const uint32_t oc = h.oc, Mc = h.Mc, n0 = h.n0, nn = h.nn;  // nn: the layer's native requests
    const bool staged = Mc <= cap;  // the same for the whole workgroup
    uint32_t *sL = sLb + bi * cap;
    const uint32_t *boff = boffb + bi * (Dk + 1);
    const uint32_t *LI = staged ? sL : A.LISTD + oc;
    if (t == 0) {
      // an issue time outside [0, 2^61) fails a layer that has requests; an
      // empty layer fails only behind a failed one (negative time)
      s_err = (tl < 0 || (any_req && tl >= ISSUE_LIMIT)) ? ERR_RANGE_TIME : 0u;
      s_last = NEG;
    }
    // the layer's issue times, a contiguous 1/C slice per workgroup; a 1/C
    // share of the native requests
    {
      const int64_t la = A.ls[l], lb = A.ls[l + 1];
      const int64_t sl = (lb - la + C - 1) / C, sa = la + (int64_t)c * sl, sb = sa + sl < lb ? sa + sl : lb;
      for (int64_t i = sa + t; i < sb; i += RBLK) A.issue[i] = tl;
    }
    for (uint32_t q = c + t * C; q < nn; q += RBLK * C) A.complete[A.LISTD[n0 + q]] = tl;
    for (uint32_t d = t; d < Dk; d += RBLK) {
      m[d] = boff[d + 1] - boff[d];
      base[d] = imax(tl, dfree[d]);
    }
    __syncthreads();
    for (uint32_t d = t; d < Dk; d += RBLK)
      if (m[d] && base[d] >= TIME_LIMIT - (int64_t)m[d] * tR) atomicOr(&s_err, ERR_OVERFLOW);
    __syncthreads();
    const bool go = s_err == 0;  // the same for the whole workgroup
    if (go) {
      for (uint32_t q = t; q < Dk * Dk; q += RBLK) {
        const uint32_t b0 = q / Dk, b1 = q - b0 * Dk;
        const int64_t delta = base[b0] - base[b1];
        const int64_t al = floor_div(delta, tR);
        const int64_t lim = int64_t(1) << 23;  // beyond any rank: clamping keeps every count
        pairs[q] = make_uint4((uint32_t)(int32_t)(al < -lim ? -lim : (al > lim ? lim : al)),
                              (uint32_t)(delta - al * tR), b0 == b1 ? 0u : m[b1], boff[b1]);
      }
      __syncthreads();
      if (staged)
        lay_rank_scan(sL, sRV, sRI, Mc, Dk, boff, base, pairs, tR, xfer, cfree, A.complete, shm, &s_chunk, &s_last,
                      &s_err);
      else
        lay_rank_scan(A.LISTD + oc, A.RV + oc, A.RI + oc, Mc, Dk, boff, base, pairs, tR, xfer, cfree, A.complete,
                      shm, &s_chunk, &s_last, &s_err);
    }
    __syncthreads();
    fetch(l + 1, 64);  // waves 1 and up, meanwhile wave 0 exchanges
    // the layer's exchange: the channel's latest completion, or its error
    if (t == 0) {
      const uint32_t e = s_err;
      const uint64_t wv = e ? (uint64_t)(1u + e) : lay_enc(Mc ? s_last : NEG);
      __hip_atomic_store(&A.SLOT[(size_t)l * C + c], wv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (t < 64) {  // wave 0 waits for every channel's word of the layer
      uint32_t anyerr = 0;
      int64_t lmax = NEG;
      for (uint32_t c1 = lane; c1 < C; c1 += 64) {
        uint64_t wv = 0;
        for (uint32_t spin = 0;; spin++) {
          wv = __hip_atomic_load(&A.SLOT[(size_t)l * C + c1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (wv) break;
          if (spin >= LAY_SPIN_ROUNDS) {  // bounded: fail the layer rather than hang
            wv = 1u + ERR_INTERNAL;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
        if (wv < LAY_VALID) anyerr |= (uint32_t)(wv - 1);
        else lmax = imax(lmax, lay_dec(wv));
      }
      anyerr = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_or(anyerr));
      lmax = wave_max(lmax);
      if (t == 0) {
        s_any = anyerr;
        s_lmax = lmax;
      }
    }
    __syncthreads();
    const uint32_t anyerr = s_any;
    const int64_t dl = anyerr ? HBF_TIME_ERROR : imax(tl, s_lmax);
    if (anyerr) {
      // the layer failed as a whole: no completion, clocks unchanged
      for (uint32_t p = t; p < Mc; p += RBLK) A.complete[LI[p]] = HBF_TIME_ERROR;
      for (uint32_t q = c + t * C; q < nn; q += RBLK * C) A.complete[A.LISTD[n0 + q]] = HBF_TIME_ERROR;
      if (t == 0 && c == 0 && any_req) atomicOr(&A.st->sticky, anyerr);
    } else {
      for (uint32_t d = t; d < Dk; d += RBLK)
        if (m[d]) dfree[d] = base[d] + (int64_t)m[d] * tR;
      if (Mc) cfree = s_last;
    }
    if (t == 0 && c == 0) A.done[l] = dl;
    prev_done = dl;
    __syncthreads();
  }
  for (uint32_t d = t; d < Dk; d += RBLK) A.st->die_free[c * Dk + d] = dfree[d];
  if (t == 0) A.st->chan_free[c] = cfree;
}

size_t lds_lay_count(uint32_t K) { return ((sizeof(LdsRanges) + 15) & ~size_t(15)) + (size_t)(K + 1) * 4; }
size_t lds_lay_place(uint32_t K) { return (size_t)(K + 1) * 4 + LWAVES * (size_t)(K + 1) * 2 + 4 + LWAVES * (size_t)(K + 1) * 4; }
size_t lds_lay_run_fixed(uint32_t Dk) {
  return (size_t)Dk * Dk * 16 + (size_t)Dk * 16 + (size_t)Dk * 4 + 2 * (Dk + 1) * 4;
}
// Staged requests per layer and channel: what the LDS holds beside the
// fixed part, at 20 bytes each (term, index by rank, two request lists), up
// to 8,192.
constexpr size_t LAY_LDS_BUDGET = 152 * 1024;
uint32_t lay_cap(uint32_t Dk) {
  const size_t f = lds_lay_run_fixed(Dk);
  const size_t c = f < LAY_LDS_BUDGET ? (LAY_LDS_BUDGET - f) / 20 : 0;
  return (uint32_t)(c > 8192 ? 8192 : c);
}
size_t lds_lay_run(uint32_t Dk) { return lds_lay_run_fixed(Dk) + (size_t)lay_cap(Dk) * 20; }

}  // namespace

// Whether the one-launch path can take a call: it needs every channel's
// workgroup resident at once (they exchange each layer's done time).
bool layers_fast_ok(const Geo &g, int ncu) {
  if (g.Dk > MAX_RUNS || g.K + 1 > 0xFFFF || g.C > 4096) return false;
  int dev = 0, coop = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop)
    return false;
  if (hipFuncSetAttribute((const void *)k_lay_run, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds_lay_run(g.Dk)) != hipSuccess ||
      hipFuncSetAttribute((const void *)k_lay_place, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds_lay_place(g.K)) != hipSuccess)
    return false;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void *)k_lay_run, RBLK, lds_lay_run(g.Dk)) !=
      hipSuccess)
    return false;
  return (int64_t)per_cu * ncu >= (int64_t)g.C;
}

// Tiles of the pre-passes: the layers cut into pieces of at most LAY_TILE
// requests (an empty layer has none).
constexpr int64_t LAY_TILE = 8192;
static uint32_t n_tiles(const int64_t *ls, int L) {
  uint64_t nt = 0;
  for (int l = 0; l < L; l++) nt += (uint64_t)((ls[l + 1] - ls[l] + LAY_TILE - 1) / LAY_TILE);
  return (uint32_t)nt;
}

size_t layers_ws_bytes(const Geo &g, int64_t n, int L) {
  const size_t KB = g.K + 1, nt = (size_t)n / LAY_TILE + L + 1;
  return 256 * 16 + (size_t)(L + 1) * 8 + (size_t)(L + 1) * 4 + nt * sizeof(LayTile) + (size_t)n * (2 + 4 + 8 + 4) +
         nt * KB * 4 * 2 + (size_t)L * (KB + 1) * 4 + (size_t)L * g.C * 8;
}

hipError_t launch_layers(const Geo &g, const RangeTable &rt, char *ws, DevState *st, const uint64_t *addr,
                         int64_t n, const int64_t *host_ls, int L, int64_t t_start, int64_t compute_ns,
                         int64_t *issue, int64_t *complete, int64_t *done, std::vector<unsigned char> &up,
                         hipEvent_t up_done, hipStream_t s) {
  const size_t KB = g.K + 1;
  const uint32_t NT = n_tiles(host_ls, L);
  // host side: the layer starts, each layer's first tile, the tile list (one
  // upload from a buffer the model keeps; an earlier call's upload must have
  // left it first)
  hipError_t e;
  if ((e = hipEventSynchronize(up_done)) != hipSuccess) return e;
  const size_t b_ls = (size_t)(L + 1) * 8, b_t0 = ((size_t)(L + 1) * 4 + 7) & ~size_t(7);
  up.resize(b_ls + b_t0 + (size_t)(NT ? NT : 1) * sizeof(LayTile));
  int64_t *h_ls = (int64_t *)up.data();
  uint32_t *h_t0 = (uint32_t *)(up.data() + b_ls);
  LayTile *h_tiles = (LayTile *)(up.data() + b_ls + b_t0);
  uint32_t q = 0;
  for (int l = 0; l < L; l++) {
    h_ls[l] = host_ls[l];
    h_t0[l] = q;
    for (int64_t a = host_ls[l]; a < host_ls[l + 1]; a += LAY_TILE)
      h_tiles[q++] = LayTile{a, a + LAY_TILE < host_ls[l + 1] ? a + LAY_TILE : host_ls[l + 1], (uint32_t)l, h_t0[l]};
  }
  h_ls[L] = host_ls[L];
  h_t0[L] = q;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    char *p = ws + o;
    o = (o + bytes + 255) & ~size_t(255);
    return p;
  };
  unsigned char *d_up = (unsigned char *)take(up.size());
  const int64_t *ls = (const int64_t *)d_up;
  const uint32_t *tile0 = (const uint32_t *)(d_up + b_ls);
  const LayTile *tiles = (const LayTile *)(d_up + b_ls + b_t0);
  uint16_t *KEY = (uint16_t *)take((size_t)n * 2);
  uint32_t *CNT = (uint32_t *)take((size_t)(NT ? NT : 1) * KB * 4);
  uint32_t *TOFF = (uint32_t *)take((size_t)(NT ? NT : 1) * KB * 4);
  uint32_t *OFF = (uint32_t *)take((size_t)L * (KB + 1) * 4);
  uint32_t *LISTD = (uint32_t *)take((size_t)n * 4);
  int64_t *RV = (int64_t *)take((size_t)n * 8);
  uint32_t *RI = (uint32_t *)take((size_t)n * 4);
  uint64_t *SLOT = (uint64_t *)take((size_t)L * g.C * 8);
  if ((e = hipMemcpyAsync(d_up, up.data(), up.size(), hipMemcpyHostToDevice, s)) != hipSuccess) return e;
  if ((e = hipEventRecord(up_done, s)) != hipSuccess) return e;
  if (NT) {
    if (g.pow2)
      hipLaunchKernelGGL(k_lay_count<true>, dim3(NT), dim3(LBLK), lds_lay_count(g.K), s, addr, tiles, g, rt, KEY, CNT);
    else
      hipLaunchKernelGGL(k_lay_count<false>, dim3(NT), dim3(LBLK), lds_lay_count(g.K), s, addr, tiles, g, rt, KEY,
                         CNT);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_lay_scan, dim3(L), dim3(LBLK), 0, s, CNT, ls, tile0, g.K, OFF, TOFF, SLOT, g.C);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (NT) {
    hipLaunchKernelGGL(k_lay_place, dim3(NT), dim3(LBLK), lds_lay_place(g.K), s, tiles, KEY, g.K, TOFF, LISTD);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  LayArgs A;
  A.ls = ls;
  A.OFF = OFF;
  A.LISTD = LISTD;
  A.RV = RV;
  A.RI = RI;
  A.SLOT = SLOT;
  A.issue = issue;
  A.complete = complete;
  A.done = done;
  A.st = st;
  A.g = g;
  A.t_start = t_start;
  A.compute_ns = compute_ns;
  A.L = (uint32_t)L;
  uint32_t cap = lay_cap(g.Dk);
  void *args[] = {&A, &cap};
  return hipLaunchCooperativeKernel((const void *)k_lay_run, dim3(g.C), dim3(RBLK), args, lds_lay_run(g.Dk), s);
}

}  // namespace hbf
