// Media variant: die page-register blocking (the die-read + channel-transfer
// path of HBFSim, arXiv 2609.09800, Section "Design", with one page register
// per die queue).  A read leaves its page in the die's register; the die
// starts no other read until that page's channel transfer has completed.
// The channel still serves pages first come first served by (die-done,
// request index).
//
// The die and channel stages are now coupled: a die's next read waits on the
// channel, whose order depends on every die's reads.  A channel and its die
// queues form an independent system, so one wave runs each channel, one lane
// per die queue.  Every die queue has at most one page pending at a time.
// The channel takes pending pages in (die-done, index) order, and a die
// reads its next request when its page has been transferred; each round of
// the loop serves the whole prefix of the ranked pending pages that no
// re-admitted page can overtake (all of them when the channel is
// saturated).  The die-order request lists come from the unblocked path's
// die stage (same ranks, same segments).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

namespace {

__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

// Wave-wide minimum with DPP row shifts (within rows of 16 by 1, 2, 4, 8,
// then row 0 -> 1, 2 -> 3 and rows 0-1 -> 2-3): lane 63 ends with the
// minimum of all 64 lanes, which readlane broadcasts.  Lanes without a
// source keep the identity.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROWMASK, 0xF, false);
}
constexpr int SHR1 = 0x111, SHR2 = 0x112, SHR4 = 0x114, SHR8 = 0x118, BC15 = 0x142, BC31 = 0x143;

// Within each row of 16 lanes, rotated right by S: lane l receives lane
// (l - S) mod 16's value, so S = 1..15 visit every other lane of the row once.
template <int S>
__device__ __forceinline__ uint32_t ror32(uint32_t x) {
  return dpp_u32<0x120 | S, 0xF>(x, x);
}
template <int S>
__device__ __forceinline__ int64_t ror64(int64_t x) {
  const uint32_t lo = ror32<S>((uint32_t)x), hi = ror32<S>((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
template <int S = 1>
__device__ __forceinline__ void row_rotations(int64_t key, uint32_t kix, int64_t (&kd)[15], uint32_t (&ki)[15]) {
  kd[S - 1] = ror64<S>(key);
  ki[S - 1] = ror32<S>(kix);
  if constexpr (S < 15) row_rotations<S + 1>(key, kix, kd, ki);
}
template <int S = 1>
__device__ __forceinline__ int64_t row_prefix_max(int64_t val, uint32_t rr, uint32_t r, int64_t M) {
  const int64_t vj = ror64<S>(val);
  const uint32_t rj = ror32<S>(rr);
  if (rj <= r) M = vj > M ? vj : M;
  if constexpr (S < 15) return row_prefix_max<S + 1>(val, rr, r, M);
  return M;
}
// minimum over the 16 lanes of row 0, broadcast
__device__ __forceinline__ uint32_t row0_min32(uint32_t x) {
  x = min(x, dpp_u32<SHR1, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR2, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR4, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR8, 0xF>(UINT32_MAX, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
}

__device__ __forceinline__ int64_t lane_i64(int64_t x, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)x >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ uint32_t wave_min32(uint32_t x) {
  x = min(x, dpp_u32<SHR1, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR2, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR4, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<SHR8, 0xF>(UINT32_MAX, x));
  x = min(x, dpp_u32<BC15, 0xA>(UINT32_MAX, x));
  x = min(x, dpp_u32<BC31, 0xC>(UINT32_MAX, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

}  // namespace

// Per lane, the die queue's upcoming requests (index, issue time) wait in an
// LDS ring of RING entries.  The next CHUNK_R of them are always in flight
// in registers: a top-up writes them to the ring and starts loading the
// following CHUNK_R, so their memory latency overlaps the steps in between
// and a step reads LDS only.  Completions (and the completion times of
// claimed refresh quanta) are staged in LDS and written out by the whole
// wave, OUTB at a time.
constexpr int RING = 64;
constexpr int CHUNK_R = 32;
constexpr int RSTRIDE = RING + 1;   // padded: lanes' rings start in different banks
constexpr int OUTB = 256;           // staged completions per write-out
constexpr int QB = 128;             // staged quantum completions per write-out

// One wave per channel (blockIdx.x); lane j = die queue c*Dk + j.
//   DDw / IX: die-ordered request indices (packed word's low half when the
//   cell shift is <= 32, else IX); issue_do: their issue times; seg_start /
//   totals: each die queue's run.  ref: refresh quanta pending (each die
//   queue's first ref_pend admissions claim one, tQ before the read; the
//   quantum's completion is written).
// ROW: at most 16 die queues per channel, all in lanes 0-15 (one DPP row),
// so the all-pairs comparisons of a round run on row rotations.
template <bool ROW>
__global__ __launch_bounds__(64) void k_regblock(const uint64_t *__restrict__ DDw, const uint32_t *__restrict__ IX,
                                                 const int64_t *__restrict__ issue_do,
                                                 const uint32_t *__restrict__ seg_start,
                                                 const uint32_t *__restrict__ totals, Geo g, DevState *st,
                                                 CallCtl *ctl, int64_t *__restrict__ complete,
                                                 int64_t *__restrict__ dfnew, int64_t *__restrict__ cfnew, int ref) {
  __shared__ uint32_t ring_idx[64 * RSTRIDE];
  __shared__ int64_t ring_iss[64 * RSTRIDE];
  __shared__ uint32_t out_idx[OUTB];
  __shared__ int64_t out_cpl[OUTB];
  __shared__ uint32_t q_die[QB], q_rank[QB];
  __shared__ int64_t q_val[QB];
  if (__hip_atomic_load(&ctl->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
  const uint32_t c = blockIdx.x, lane = __lane_id(), Dk = g.Dk;
  const bool on = lane < Dk;
  const uint32_t k = c * Dk + (on ? lane : 0);
  const bool narrow = ctl->shift <= 32;
  const int64_t tR = g.tR, tQ = g.tQ, xfer = g.xfer;
  const uint32_t total = on ? totals[k] : 0;
  const uint32_t base = on ? seg_start[k] : 0;
  const uint32_t R = (on && ref) ? st->ref_pend[k] : 0;
  int64_t free_at = on ? st->die_free[k] : NEG;  // NEG: idle since minus infinity
  int64_t cfree = st->chan_free[c];              // NEG: idle since minus infinity
  uint32_t err = 0;

  auto lds_sync = [&]() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  // request indices: the low half of each packed die-order word, or IX
  const uint32_t *ixs = narrow ? reinterpret_cast<const uint32_t *>(DDw) : IX;
  const uint32_t ixstride = narrow ? 2u : 1u;
  uint32_t loaded = 0;     // requests of this die queue written to the ring
  uint32_t admitted = 0;   // requests whose read has been scheduled
  uint32_t nix[CHUNK_R];   // in flight: requests loaded .. loaded + CHUNK_R - 1
  int64_t nis[CHUNK_R];
  auto fetch = [&]() {     // per lane: start loading the chunk after `loaded`
#pragma unroll
    for (int j = 0; j < CHUNK_R; j++) {
      const uint32_t r = loaded + j;
      const bool v = on && r < total;
      nix[j] = ixs[v ? (size_t)(base + r) * ixstride : 0];
      nis[j] = issue_do[v ? base + r : 0];
    }
  };
  // wave-uniform: every lane whose ring has room for the chunk in flight
  // writes it and starts the next one
  auto top_up = [&]() {
    const bool go = on && loaded < total && loaded - admitted <= (uint32_t)(RING - CHUNK_R);
    if (go) {
#pragma unroll
      for (int j = 0; j < CHUNK_R; j++) {
        const uint32_t r = loaded + j;
        if (r < total) {
          ring_idx[lane * RSTRIDE + r % RING] = nix[j];
          ring_iss[lane * RSTRIDE + r % RING] = nis[j];
        }
      }
      loaded = min(total, loaded + CHUNK_R);
      fetch();
    }
    lds_sync();
  };

  uint32_t nout = 0, nq = 0;   // staged completions / quantum completions (uniform)
  auto flush_out = [&]() {     // wave-uniform
    lds_sync();
    for (uint32_t j = lane; j < nout; j += 64) complete[out_idx[j]] = out_cpl[j];
    nout = 0;
    lds_sync();
  };
  auto flush_q = [&]() {       // wave-uniform
    lds_sync();
    for (uint32_t j = lane; j < nq; j += 64) {
      const uint32_t kk = q_die[j];
      *st->ref_slot[st->ref_off[kk] + st->ref_head[kk] + q_rank[j]] = q_val[j];
    }
    nq = 0;
    lds_sync();
  };

  int64_t dd = INT64_MAX;  // die-done of the pending page
  uint32_t pidx = UINT32_MAX;
  // the die reads its next request; returns whether it claimed a quantum
  auto admit = [&]() -> bool {
    const uint32_t sl = lane * RSTRIDE + admitted % RING;
    const bool claim = admitted < R;
    int64_t s0 = max64(ring_iss[sl], free_at);
    if (claim) s0 += tQ;
    dd = s0 + tR;
    pidx = ring_idx[sl];
    if (dd >= TIME_LIMIT) err |= ERR_OVERFLOW;
    admitted++;
    return claim;
  };
  fetch();
  top_up();
  {  // every die queue's first read; claims staged in lane order
    const bool cl = total ? admit() : false;
    const uint64_t cm = __ballot(cl);
    if (cl) {
      const uint32_t slot = (uint32_t)__popcll(cm & ((1ull << lane) - 1));
      q_die[slot] = k;
      q_rank[slot] = 0;
      q_val[slot] = dd - tR;
    }
    nq = (uint32_t)__popcll(cm);
    if (nq) flush_q();
  }
  top_up();   // second chunk into the ring, third in flight
  // each die queue's next request (after the pending one), read from its
  // ring a round ahead of its use
  int64_t nx_iss = 0;
  uint32_t nx_idx = UINT32_MAX;
  if (on && admitted < total) {
    const uint32_t sl = lane * RSTRIDE + admitted % RING;
    nx_iss = ring_iss[sl];
    nx_idx = ring_idx[sl];
  }

  // Rounds.  Every die queue with a page pending is ranked by (die-done,
  // index).  If the channel takes the pending pages in that order, the page
  // of rank r completes at (r+1)*xfer + max(cfree, max over ranks i <= r of
  // die_done_i - i*xfer), and its die can then read its next request.  The
  // channel really does take them in that order up to the first rank that
  // some die's next page (read after an earlier rank's transfer) would
  // precede; that prefix is served at once, its dies are re-admitted, and
  // the next round ranks again.  A saturated channel serves every pending
  // page per round; an idle one at least the first.
  uint32_t left = total;             // not yet transferred
  bool any = false;
  for (;;) {
    const bool pend = left != 0;
    const uint64_t pm = __ballot(pend);
    if (pm == 0) break;
    const uint32_t P = (uint32_t)__popcll(pm);
    // rank among the pending pages (other lanes' pages: key INT64_MAX)
    const int64_t key = pend ? dd : INT64_MAX;
    const uint32_t kix = pend ? pidx : UINT32_MAX;
    int64_t kd[15];
    uint32_t ki[15];
    uint32_t r = 0;
    if (ROW) {
      row_rotations(key, kix, kd, ki);
#pragma unroll
      for (int q = 0; q < 15; q++) r += (kd[q] < key || (kd[q] == key && ki[q] < kix)) ? 1u : 0u;
    } else {
      for (uint64_t mm = pm; mm; mm &= mm - 1) {
        const int j = (int)__builtin_ctzll(mm);
        const int64_t dj = lane_i64(dd, j);
        const uint32_t ij = (uint32_t)__builtin_amdgcn_readlane((int)pidx, j);
        r += (dj < dd || (dj == dd && ij < pidx)) ? 1u : 0u;
      }
    }
    // completion if every lower rank is served first
    const int64_t val = dd - (int64_t)r * xfer;
    int64_t M = max64(cfree, val);
    if (ROW) {
      M = row_prefix_max(val, pend ? r : 0xFFFFu, r, M);
    } else {
      for (uint64_t mm = pm; mm; mm &= mm - 1) {
        const int j = (int)__builtin_ctzll(mm);
        const int64_t vj = lane_i64(val, j);
        const uint32_t rj = (uint32_t)__builtin_amdgcn_readlane((int)r, j);
        if (rj <= r) M = max64(M, vj);
      }
    }
    const int64_t cpl = (int64_t)(r + 1) * xfer + M;
    // the die's next read once this page has left its register
    bool claim = false;
    int64_t ndd = INT64_MAX;
    uint32_t nidx = UINT32_MAX;
    if (pend && admitted < total) {
      claim = admitted < R;
      int64_t s0 = max64(nx_iss, cpl);
      if (claim) s0 += tQ;
      ndd = s0 + tR;
      nidx = nx_idx;
    }
    // first rank that this next page would precede
    uint32_t cut = P;
    if (ROW) {
      uint32_t c2 = 1;  // its own pending page precedes it
#pragma unroll
      for (int q = 0; q < 15; q++) c2 += (kd[q] < ndd || (kd[q] == ndd && ki[q] < nidx)) ? 1u : 0u;
      if (ndd != INT64_MAX) cut = c2;
    } else if (ndd != INT64_MAX) {
      cut = 0;
      for (uint64_t mm = pm; mm; mm &= mm - 1) {
        const int j = (int)__builtin_ctzll(mm);
        const int64_t dj = lane_i64(dd, j);
        const uint32_t ij = (uint32_t)__builtin_amdgcn_readlane((int)pidx, j);
        cut += (dj < ndd || (dj == ndd && ij < nidx)) ? 1u : 0u;
      }
    }
    // >= 1: a next page follows its own
    const uint32_t v = ROW ? row0_min32(pend ? cut : UINT32_MAX) : wave_min32(pend ? cut : UINT32_MAX);
    const bool served = pend && r < v;
    if (served) {
      out_idx[nout + r] = pidx;
      out_cpl[nout + r] = cpl;
      left--;
      free_at = cpl;  // the page has left the register
      if (cpl >= TIME_LIMIT) err |= ERR_OVERFLOW;
    }
    const uint64_t last = __ballot(served && r == v - 1);
    cfree = lane_i64(cpl, (int)__builtin_ctzll(last));
    any = true;
    nout += v;
    const bool adm = served && left != 0;
    if (adm) {
      dd = ndd;
      pidx = nidx;
      admitted++;
      if (dd >= TIME_LIMIT) err |= ERR_OVERFLOW;
    }
    const bool cl = adm && claim;
    const uint64_t cm = __ballot(cl);
    if (cm) {
      if (cl) {
        const uint32_t slot = nq + (uint32_t)__popcll(cm & ((1ull << lane) - 1));
        q_die[slot] = k;
        q_rank[slot] = admitted - 1;
        q_val[slot] = dd - tR;
      }
      nq += (uint32_t)__popcll(cm);
      if (nq > QB - 64) flush_q();
    }
    if (nout > OUTB - 64) flush_out();
    // Steady rounds.  If this round served every pending page back to back
    // and every die re-read at once (its next request issued by then, no
    // quantum claimed), the next round ranks the dies in the same order:
    // each next page is ready tR after its predecessor left, and with
    // P*xfer >= tR + xfer it is ready before the channel reaches it.  So
    // in round j = 1, 2, ... the page of rank r completes at
    // cf + ((j-1)*P + r + 1)*xfer, as long as every die's page of that round
    // was issued by its predecessor's completion and claims nothing.  Each
    // lane checks its own queue ahead, the shortest run decides, and those
    // rounds are written at once; the round after them is admitted as usual.
    const bool steady = v == P && cm == 0 && (int64_t)P * xfer >= tR + xfer && !__ballot(pend && !adm) &&
                        !__ballot(pend && (cpl != cfree - (int64_t)(P - 1 - r) * xfer || dd != cpl + tR));
    if (steady) {
      constexpr uint32_t FL = 16, FMAX = 4096;  // rounds per lane per batch, rounds per step
      const int64_t cf0 = cfree;
      const uint32_t a0 = admitted;             // the pending page is request a0 - 1 of the queue
      // Every lane works here: lane l takes die queue l mod Dp (Dp: Dk
      // rounded up to a power of two) and every S-th round (S = 64 / Dp),
      // so a batch covers S*FL rounds.  Per batch: load each round's request
      // (issue time, index), find the first round some die cannot keep,
      // write the rounds before it.
      const uint32_t lgD = Dk <= 16 ? 4u : Dk <= 32 ? 5u : 6u, S = 64u >> lgD;
      const uint32_t dl = lane & ((1u << lgD) - 1), sub = lane >> lgD;
      const bool pd = __shfl((int)(pend ? 1 : 0), (int)dl) != 0;
      const uint32_t a0d = (uint32_t)__shfl((int)a0, (int)dl), rd = (uint32_t)__shfl((int)r, (int)dl);
      const uint32_t td = (uint32_t)__shfl((int)total, (int)dl), Rd = (uint32_t)__shfl((int)R, (int)dl);
      const uint32_t bd = (uint32_t)__shfl((int)base, (int)dl);
      uint32_t m = 0;                           // rounds written (round 1: the pending pages)
      for (uint32_t j0 = 1;; j0 += S * FL) {
        uint32_t bad = UINT32_MAX;
        int64_t is[FL];
        uint32_t ix[FL];
        if (pd) {
#pragma unroll
          for (uint32_t u = 0; u < FL; u++) {
            const uint32_t pos = a0d + j0 + sub + S * u - 2, at = pos < td ? bd + pos : bd;
            is[u] = issue_do[at];
            ix[u] = ixs[(size_t)at * ixstride];
          }
#pragma unroll
          for (int u = (int)FL - 1; u >= 0; u--) {
            const uint32_t j = j0 + sub + S * (uint32_t)u, pos = a0d + j - 2;
            const bool ok = j == 1 || (pos < td && pos >= Rd &&
                                       is[u] <= cf0 + ((int64_t)(j - 2) * P + rd + 1) * xfer);
            if (!ok) bad = j;
          }
        }
        const uint32_t fb = wave_min32(bad);
        const uint32_t upto = fb == UINT32_MAX ? j0 + S * FL - 1 : fb - 1;
        if (pd) {
#pragma unroll
          for (uint32_t u = 0; u < FL; u++) {
            const uint32_t j = j0 + sub + S * u;
            if (j <= upto) complete[ix[u]] = cf0 + ((int64_t)(j - 1) * P + rd + 1) * xfer;
          }
        }
        m = upto;
        if (fb != UINT32_MAX || m >= FMAX) break;
      }
      const int64_t clm = cf0 + ((int64_t)(m - 1) * P + r + 1) * xfer;  // this lane's last completion
      cfree = cf0 + (int64_t)m * P * xfer;
      bool cl2 = false;
      if (pend) {
        if (clm >= TIME_LIMIT) err |= ERR_OVERFLOW;
        left -= m;
        free_at = clm;
        if (left != 0) {  // admit the page of round m + 1
          const uint32_t pos = a0 + m - 1;
          cl2 = pos < R;
          int64_t s0 = max64(issue_do[base + pos], clm);
          if (cl2) s0 += tQ;
          dd = s0 + tR;
          pidx = ixs[(size_t)(base + pos) * ixstride];
          admitted = pos + 1;
          if (dd >= TIME_LIMIT) err |= ERR_OVERFLOW;
        }
      }
      const uint64_t cm2 = __ballot(cl2);
      if (cm2) {
        if (cl2) {
          const uint32_t slot = nq + (uint32_t)__popcll(cm2 & ((1ull << lane) - 1));
          q_die[slot] = k;
          q_rank[slot] = admitted - 1;
          q_val[slot] = dd - tR;
        }
        nq += (uint32_t)__popcll(cm2);
        if (nq > QB - 64) flush_q();
      }
      // the ring restarts after the requests admitted here
      if (pend && loaded < admitted) {
        loaded = admitted;
        fetch();
      }
      top_up();
      if (pend && left != 0 && admitted < total) {
        const uint32_t sl = lane * RSTRIDE + admitted % RING;
        nx_iss = ring_iss[sl];
        nx_idx = ring_idx[sl];
      }
      continue;
    }
    // each die's next request must be in its ring before the next round
    if (__ballot(on && admitted < total && loaded - admitted < 2)) top_up();
    if (adm && admitted < total) {
      const uint32_t sl = lane * RSTRIDE + admitted % RING;
      nx_iss = ring_iss[sl];
      nx_idx = ring_idx[sl];
    }
  }
  if (nout) flush_out();
  if (nq) flush_q();
  if (on && total) dfnew[k] = free_at;
  if (lane == 0) {
    cfnew[c] = cfree;
    if (any) atomicMax((long long *)&ctl->max_cpl, (long long)cfree);
  }
  if (__ballot(err != 0)) {
    uint32_t e = err;
    for (int d = 32; d >= 1; d >>= 1) e |= (uint32_t)__shfl_xor((int)e, d);
    if (lane == 0) atomicOr(&ctl->err, e);
  }
}

hipError_t launch_regblock(const Geo &g, const uint64_t *DDw, const uint32_t *IX, const int64_t *issue_do,
                           const uint32_t *seg_start, const uint32_t *totals, DevState *st, CallCtl *ctl,
                           int64_t *complete, int64_t *dfnew, int64_t *cfnew, bool ref, hipStream_t s) {
  hipLaunchKernelGGL(g.Dk <= 16 ? k_regblock<true> : k_regblock<false>, dim3(g.C), dim3(64), 0, s, DDw, IX,
                     issue_do, seg_start, totals, g, st, ctl, complete, dfnew, cfnew, ref ? 1 : 0);
  return hipGetLastError();
}

}  // namespace hbf
