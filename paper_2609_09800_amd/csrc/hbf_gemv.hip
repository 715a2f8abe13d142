// Instrumented bf16 grouped GEMV with HBF delay injection at consumption.
//
// HBFSim (arXiv 2609.09800, Section "D2: Preserving GPU Asynchrony") splits
// an access into issue and consumption: after issuing a load the program
// continues, and the modeled latency is charged only at the first use of the
// loaded value.  Here a workgroup issues every load of a weight page and
// only then waits -- right before the first multiply that consumes the data
// -- until the page's modeled completion.  Waits are measured on the GPU's
// constant-rate wall clock (s_memrealtime); no host clock is involved, so no
// clock origins are mixed.
//
// One time origin per call.  Every page of a call is issued at the call's
// start, so page q is released at origin + (complete[q] - issue[q]), where
// origin is the wall clock at which the consuming kernel began: a first
// one-thread kernel clears the origin record, the timed kernel's workgroup
// 0 (dispatched first) writes its start clock there as its first act, and
// every other workgroup reads it once, at its first consumption point
// (waiting, boundedly, in the rare case it is not there yet).
// A clock taken by a separate earlier kernel would also charge the gap
// until the host has queued the timed kernel; an atomic minimum taken by
// every workgroup serializes them on one address for microseconds.  With
// delays, the call runs on persistent workgroups (at most as many as the
// GPU holds at once, so none starts late behind a waiting one), each taking
// its pages in ascending delay order; a last kernel turns the recorded
// release clocks into delays from the final origin.
//
// Y[e][b][n] = sum_k X[e][b][k] * W[e][n][k], bf16 inputs, fp32 accumulate.
// Bandwidth bound (B flop per weight byte).  Delayed calls compute page by
// page, each after its own wait, with packed bf16 dot instructions (two
// products per instruction, fp32 accumulate); calls without delays have no
// consumption point to honour and take the matrix cores on 16-row tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

constexpr int GEMV_MAXV = 8;  // 16-byte weight vectors held per lane
// Longest wait of a workgroup for the call's origin (never reached: workgroup
// 0 publishes it as soon as it starts); past it the call fails.
constexpr int64_t ORIGIN_WAIT_PS = 100000000000;  // 100 ms
// Longest delay one page may inject; longer requests are clamped to it and
// reported (HBF_ERANGE_TIME) so that a bad time array can never stall the GPU.
constexpr int64_t MAX_PAGE_DELAY_NS = 1000000000;
// Pages one persistent workgroup may take (one per thread when ordering).
constexpr int GEMV_MAXP = 256;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t w, uint32_t x, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), __builtin_bit_cast(bf16x2_t, x), acc,
                                         false);
}

// 8 bf16 products summed in fp32 (four packed two-product dot instructions)
__device__ __forceinline__ float dot8(uint4 w, uint4 x) {
  float s = dot2(w.x, x.x, 0.0f);
  s = dot2(w.y, x.y, s);
  s = dot2(w.z, x.z, s);
  s = dot2(w.w, x.w, s);
  return s;
}

// ------------------------------------------------------------------ timing

// Wall-clock ticks page q must wait: ceil((complete - issue) / tick).  Times
// outside [0, 2^62) or a completion before the issue are errors (no wait,
// HBF_ERANGE_TIME); delays above MAX_PAGE_DELAY_NS are clamped and reported.
__device__ __forceinline__ uint64_t page_ticks(const int64_t *pi, const int64_t *pc, int q, int64_t tick_ps,
                                               uint32_t *errb) {
  const int64_t a = pi[q], b = pc[q];
  if (a < 0 || b < 0 || a >= TIME_LIMIT || b >= TIME_LIMIT || b < a) {
    *errb |= ERR_RANGE_TIME;
    return 0;
  }
  int64_t d = b - a;
  if (d > MAX_PAGE_DELAY_NS) {
    d = MAX_PAGE_DELAY_NS;
    *errb |= ERR_RANGE_TIME;
  }
  return (uint64_t)((d * 1000 + tick_ps - 1) / tick_ps);
}

// The call's origin as published by the timed kernel's workgroup 0, waiting
// (boundedly) until it is there; past the bound the caller's own clock
// stands in and the call fails with ERR_INTERNAL.
__device__ __forceinline__ uint64_t read_origin(DevState *st, int64_t tick_ps, uint32_t *errb) {
  const uint64_t start = __builtin_amdgcn_s_memrealtime();
  const uint64_t limit = (uint64_t)(ORIGIN_WAIT_PS / tick_ps);
  uint64_t o = __hip_atomic_load(&st->gemv_origin, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
  while (o == ~uint64_t(0)) {
    if (__builtin_amdgcn_s_memrealtime() - start > limit) {
      *errb |= ERR_INTERNAL;
      return start;
    }
    __builtin_amdgcn_s_sleep(2);
    o = __hip_atomic_load(&st->gemv_origin, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
  }
  return o;
}

// Consumption point of a delayed page: spin until `ticks` have passed since
// the call's origin.  Returns the release clock.
__device__ __forceinline__ uint64_t wait_release(uint64_t origin, uint64_t ticks) {
  uint64_t now = __builtin_amdgcn_s_memrealtime();
  while (now < origin || now - origin < ticks) {  // (a clock read below the origin waits too)
    __builtin_amdgcn_s_sleep(1);
    now = __builtin_amdgcn_s_memrealtime();
  }
  return now;
}

// First kernel of a delayed call: clears its origin record (the timed
// kernel's workgroup 0 writes its start clock there).
__global__ void k_gemv_origin(DevState *st) {
  if (threadIdx.x == 0) st->gemv_origin = ~uint64_t(0);
}

// Last kernel of a delayed call with measurements: release clock -> delay
// from the origin, in ns.
__global__ __launch_bounds__(256) void k_gemv_measured(int64_t *__restrict__ meas, int npages, int64_t tick_ps,
                                                       const DevState *st) {
  const uint64_t o = st->gemv_origin;
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q < npages) {
    const uint64_t rel = (uint64_t)meas[q];
    meas[q] = rel < o ? 0 : (int64_t)((rel - o) * (uint64_t)tick_ps / 1000);
  }
}

// ------------------------------------------------------------------ page bodies

// General shape: one page of R = page_bytes / (2K) rows by one 256-thread
// workgroup.  Wave w takes rows w, w+4, ...; lane l takes the 16-byte
// vectors l, l+64, ... of each row (VPL = K/512 of them).  `wait` runs
// between the page's loads and its first use.
template <typename Wait>
__device__ __forceinline__ void page_general(int q, const uint16_t *__restrict__ W, int K, int N, int R,
                                             const uint16_t *__restrict__ X, int B, float *__restrict__ Y,
                                             Wait wait) {
  const int row0 = q * R;
  const int e = row0 / N;
  const int nb = row0 - e * N;
  const int VPL = K >> 9;
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int RPW = (R + 3) >> 2;

  // ---- issue: every load of this page
  uint4 v[GEMV_MAXV];
#pragma unroll
  for (int s = 0; s < GEMV_MAXV; s++) {
    const int rw = s / VPL, tv = s - rw * VPL;
    const int rl = w + 4 * rw;
    if (rw < RPW && rl < R)
      v[s] = *(const uint4 *)(W + (size_t)(row0 + rl) * K + (size_t)(lane + 64 * tv) * 8);
    else
      v[s] = make_uint4(0, 0, 0, 0);
  }
  // ---- consumption point
  wait();

  // ---- consume
  const uint16_t *xe = X + (size_t)e * B * K;
  for (int b = 0; b < B; b++) {
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < GEMV_MAXV; s++) {
      const int rw = s / VPL, tv = s - rw * VPL;
      if (rw < RPW && rw < 4) {
        const uint4 xv = *(const uint4 *)(xe + (size_t)b * K + (size_t)(lane + 64 * tv) * 8);
        const float t = dot8(v[s], xv);
        if (rw == 0) part[0] += t;
        else if (rw == 1) part[1] += t;
        else if (rw == 2) part[2] += t;
        else part[3] += t;
      }
    }
#pragma unroll
    for (int rw = 0; rw < 4; rw++) {
      float t = part[rw];
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o);
      const int rl = w + 4 * rw;
      if (rw < RPW && rl < R && lane == 0) Y[((size_t)e * B + b) * N + nb + rl] = t;
    }
  }
}

// Transposing butterfly over the 64 lanes of a wave on C values per lane,
// in six steps that pair each lane with lane ^ 32, ^ 16, ^ 15, ^ 7, ^ 2 and
// ^ 1 (the masks span all six lane bits, so every lane's result sums all 64
// lanes).  While a lane has more than one value, a step halves them: the
// lane keeps the upper half if its decision bit (5, 4, 3, 2, 1, 0 in step
// order) is set, the lower half if not, and adds the partner's copy of that
// half.  The first two steps use gfx950's cross-row swaps, which hand each
// lane exactly the partner's copy of the half it keeps (no selects); the
// others use DPP lane permutations (row mirror, half-row mirror, quad
// permutes).  Once one value is left the remaining steps are plain sums.
// Afterwards the lane holds the wave sum of value index lane >> (6 - log2 C).
__device__ __forceinline__ float swap_sum(float a, float b, int step) {
  const auto r = step == 0 ? __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false)
                           : __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int STEP>
__device__ __forceinline__ float partner(float v) {
  return dpp_f<STEP == 2 ? 0x140 : STEP == 3 ? 0x141 : STEP == 4 ? 0x4E : 0xB1>(v);
}
template <int C, int STEP>
__device__ __forceinline__ void butterfly(float *val, int lane) {
  if constexpr (STEP < 6) {
    if constexpr (C > 1) {
      constexpr int H = C / 2;
      if constexpr (STEP < 2) {
#pragma unroll
        for (int i = 0; i < H; i++) val[i] = swap_sum(val[i], val[i + H], STEP);
      } else {
        const bool up = ((lane >> (5 - STEP)) & 1) != 0;
#pragma unroll
        for (int i = 0; i < H; i++) {
          const float lo = val[i] + partner<STEP>(val[i]);
          const float hi = val[i + H] + partner<STEP>(val[i + H]);
          val[i] = up ? hi : lo;
        }
      }
      butterfly<H, STEP + 1>(val, lane);
    } else {
      if constexpr (STEP < 2)
        val[0] = swap_sum(val[0], val[0], STEP);
      else
        val[0] += partner<STEP>(val[0]);
      butterfly<1, STEP + 1>(val, lane);
    }
  }
}

// The expert shape of the MoE workloads (K = 2048, 16 KiB pages of 4 rows)
// at batch B <= BB, BB = 1, 2, 4, 8 or 16 (rows b >= B are zero and not
// written).  Thread t of the page's workgroup holds the 16-byte column slice
// t of all 4 rows and of every activation row, so each activation vector is
// read once per workgroup (not once per row) and feeds 4 dot products.  The
// activations are loaded right after the page, before the wait.  The 4*BB
// partial sums of a lane are reduced across the wave by a transposing
// butterfly (63 exchanges for 64 values instead of 6 per value, all in
// registers), then across the 4 waves through LDS.  (Workgroups of 2 or 4
// pages, sharing one activation load, measured slower at every batch: fewer
// workgroups in flight.)
template <int BB, bool PAD, typename Wait>
__device__ __forceinline__ void page_k2048(int q, const uint16_t *__restrict__ W, int N,
                                           const uint16_t *__restrict__ X, int B_, float *__restrict__ Y,
                                           float (*red)[64], Wait wait) {
  constexpr int K = 2048, R = 4, V = R * BB;
  constexpr int LGV = V == 4 ? 2 : V == 8 ? 3 : V == 16 ? 4 : V == 32 ? 5 : 6;
  const int row0 = q * R;
  const int e = row0 / N;
  const int nb = row0 - e * N;
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;

  // ---- issue: every load of this page, then the activations
  uint4 v[R];
#pragma unroll
  for (int r = 0; r < R; r++) v[r] = *(const uint4 *)(W + (size_t)(row0 + r) * K + (size_t)t * 8);
  const int B = PAD ? B_ : BB;  // the batch (PAD: B_ < BB rows, the rest zero)
  const uint16_t *xe = X + (size_t)e * B * K + (size_t)t * 8;
  uint4 xv[BB];
#pragma unroll
  for (int b = 0; b < BB; b++) xv[b] = b < B ? *(const uint4 *)(xe + (size_t)b * K) : make_uint4(0, 0, 0, 0);

  // ---- consumption point
  wait();

  // ---- consume: value index r*BB + b
  float val[V];
#pragma unroll
  for (int b = 0; b < BB; b++)
#pragma unroll
    for (int r = 0; r < R; r++) val[r * BB + b] = dot8(v[r], xv[b]);
  butterfly<V, 0>(val, lane);
  red[w][lane] = val[0];
  __syncthreads();
  // the lane holding value index i has i's bits in its top log2(V) bits
  if (t < V) {
    const int src = t << (6 - LGV);
    const float sum = red[0][src] + red[1][src] + red[2][src] + red[3][src];
    const int r = t / BB, b = t - r * BB;
    if (b < B) Y[((size_t)e * B + b) * N + nb + r] = sum;
  }
  __syncthreads();  // red is reused by the workgroup's next page
}

// ------------------------------------------------------------------ matrix cores

// No delays, batch 9..16 (below that the per-page kernel, whose 1,536
// small workgroups stream the weights faster, measured 6.0 against 8.2 us
// per 24 MiB call at batch 1), N % 16 == 0, K % 512 == 0: one workgroup of
// 4 waves per tile of 16 weight rows (one expert's), wave w taking the K/4
// wide slice w.  Each 32-wide step of k is one v_mfma_f32_16x16x32_bf16
// with A = the expert's activations (16 rows; rows >= B are zero) and B =
// the tile's rows transposed: lane l holds 8 consecutive k of activation
// row l % 16 and, for the same k, of tile row l % 16 (k group l / 16), and
// accumulates outputs (batch 4 (l / 16) + j, tile row l % 16), j < 4.  A
// round issues KS steps' loads (16 bytes of W and of X per lane each)
// before its first product.  The slices' partial tiles meet in LDS.  At
// B < 16 the unused rows cost matrix-core cycles only (no memory traffic),
// which the instruction rate covers many times over.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma_bf16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 c, 0, 0, 0);
}

template <int KS>
__global__ __launch_bounds__(256) void k_gemv_mfma(const uint16_t *__restrict__ W, int K, int N,
                                                   const uint16_t *__restrict__ X, int B,
                                                   float *__restrict__ Y) {
  __shared__ f32x4_t red[3][64];
  const int row0 = blockIdx.x * 16;
  const int e = row0 / N, nb = row0 - e * N;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, kg = lane >> 4;
  const int kq = K >> 2;
  const uint16_t *wp = W + (size_t)(row0 + col) * K + (size_t)w * kq + kg * 8;
  const bool xon = col < B;
  const uint16_t *xp = X + ((size_t)e * B + (xon ? col : 0)) * K + (size_t)w * kq + kg * 8;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < kq; k0 += 32 * KS) {
    uint4 wv[KS], xv[KS];
#pragma unroll
    for (int s = 0; s < KS; s++) wv[s] = *(const uint4 *)(wp + k0 + 32 * s);
#pragma unroll
    for (int s = 0; s < KS; s++) xv[s] = xon ? *(const uint4 *)(xp + k0 + 32 * s) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int s = 0; s < KS; s++) acc = mfma_bf16(xv[s], wv[s], acc);
  }
  if (w) red[w - 1][lane] = acc;
  __syncthreads();
  if (w == 0) {
    acc += red[0][lane];
    acc += red[1][lane];
    acc += red[2][lane];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int b = 4 * kg + j;
      if (b < B) Y[((size_t)e * B + b) * N + nb + col] = acc[j];
    }
  }
}

// The expert shape (K = 2048) at batch 9..16: two tiles of one expert per
// workgroup of 8 waves, waves 4h .. 4h+3 on tile h as above; the second
// tile holds T1 rows (16, or 8 with its other lanes' weights zero, so that
// E*N/24 workgroups fill every CU where E*N/32 would leave some idle).
// The activation slices, the same for both tiles, are loaded once per
// workgroup into LDS (each wave fetching half of its slice's 16 steps) and
// read back in the operand layout: a quarter of the activation traffic of
// one tile per 4 waves.  Measured at batch 16 on 8 x [768 x 2048]: 9.05 us
// per call with 24 rows per workgroup (256 workgroups), 9.3 with 32 rows
// (192, before the loads were reordered), 10.9 with one tile per
// workgroup, 12.0 for the per-page kernel.
template <int T1>
__global__ __launch_bounds__(512) void k_gemv_mfma_2t(const uint16_t *__restrict__ W, int N,
                                                      const uint16_t *__restrict__ X, int B,
                                                      float *__restrict__ Y) {
  constexpr int K = 2048, KQ = K / 4, STEPS = KQ / 32, ROWS = 16 + T1;
  __shared__ uint4 xs[4][STEPS][64];  // [slice][step][lane], 64 KiB
  __shared__ f32x4_t red[2][3][64];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = w >> 2, wq = w & 3;
  const int base = blockIdx.x * ROWS;
  const int e = base / N, nb = base - e * N;  // every row lies in expert e (N % ROWS == 0)
  const int col = lane & 15, kg = lane >> 4;
  const bool won = h == 0 || col < T1;        // a row of this workgroup
  // Lanes past the tile's rows or the batch load a duplicate row (the same
  // lines as a neighbouring lane) instead of selecting zeros, so that no
  // load is waited for before the activations go to LDS; their outputs
  // (batch b depends on activation row b only) are not stored.
  const uint16_t *wp = W + (size_t)(base + h * 16 + (won ? col : col - T1)) * K + wq * KQ + kg * 8;
  const uint16_t *xp = X + ((size_t)e * B + (col < B ? col : B - 1)) * K + wq * KQ + kg * 8;
  // activation loads first, then the weights, so that both are in flight
  // when the activations are written to LDS
  uint4 xv[STEPS / 2], wv[STEPS];
#pragma unroll
  for (int i = 0; i < STEPS / 2; i++) xv[i] = *(const uint4 *)(xp + 32 * (h * (STEPS / 2) + i));
#pragma unroll
  for (int s = 0; s < STEPS; s++) wv[s] = *(const uint4 *)(wp + 32 * s);
#pragma unroll
  for (int i = 0; i < STEPS / 2; i++) xs[wq][h * (STEPS / 2) + i][lane] = xv[i];
  __syncthreads();
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < STEPS; s++) acc = mfma_bf16(xs[wq][s][lane], wv[s], acc);
  if (wq) red[h][wq - 1][lane] = acc;
  __syncthreads();
  if (wq == 0) {
    acc += red[h][0][lane];
    acc += red[h][1][lane];
    acc += red[h][2][lane];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int b = 4 * kg + j;
      if (b < B && won) Y[((size_t)e * B + b) * N + nb + h * 16 + col] = acc[j];
    }
  }
}

// ------------------------------------------------------------------ schedulers

// No delays: one workgroup per page, no clock reads.
__global__ __launch_bounds__(256) void k_gemv_general(const uint16_t *__restrict__ W, int K, int N, int R,
                                                      const uint16_t *__restrict__ X, int B,
                                                      float *__restrict__ Y) {
  page_general(blockIdx.x, W, K, N, R, X, B, Y, [] {});
}

template <int BB, bool PAD>
__global__ __launch_bounds__(256) void k_gemv_k2048(const uint16_t *__restrict__ W, int N,
                                                    const uint16_t *__restrict__ X, int B_,
                                                    float *__restrict__ Y) {
  __shared__ float red[4][64];
  page_k2048<BB, PAD>(blockIdx.x, W, N, X, B_, Y, red, [] {});
}

// With delays: persistent workgroups.  Workgroup g owns pages g + i*G
// (i < m <= GEMV_MAXP, G = gridDim.x) and serves them in ascending order of
// their wait (ties by page).  `page(q, wait)` runs one page.
template <typename Page>
__device__ __forceinline__ void timed_pages(int npages, const int64_t *__restrict__ pi,
                                            const int64_t *__restrict__ pc, int64_t *__restrict__ meas,
                                            int64_t tick_ps, DevState *st, Page page) {
  __shared__ uint64_t s_ticks[GEMV_MAXP];
  __shared__ int s_order[GEMV_MAXP];
  __shared__ uint64_t s_origin;
  const int t = threadIdx.x;
  const int G = gridDim.x, g = blockIdx.x;
  const int m = (npages - g + G - 1) / G;
  uint32_t errb = 0;
  if (g == 0 && t == 0) {  // the call's origin: workgroup 0's start, published for the others
    const uint64_t now = __builtin_amdgcn_s_memrealtime();
    __hip_atomic_store(&st->gemv_origin, now, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    s_origin = now;
  }
  uint64_t mine = 0;
  if (t < m) {
    mine = page_ticks(pi, pc, g + t * G, tick_ps, &errb);
    s_ticks[t] = mine;
  }
  __syncthreads();
  if (t < m) {  // rank among the workgroup's pages by (ticks, position)
    int r = 0;
    for (int j = 0; j < m; j++) {
      const uint64_t o = s_ticks[j];
      r += (o < mine || (o == mine && j < t)) ? 1 : 0;
    }
    s_order[r] = t;
  }
  __syncthreads();
  // other workgroups read the origin at their first delayed page's
  // consumption point, by when workgroup 0 has long published it (they wait
  // for it otherwise)
  uint64_t origin = g == 0 ? s_origin : ~uint64_t(0);
  for (int i = 0; i < m; i++) {
    const int li = s_order[i];
    const int q = g + li * G;
    const uint64_t ticks = s_ticks[li];
    page(q, [&] {
      // a page without delay is released at once and needs no origin
      if (ticks != 0 && origin == ~uint64_t(0)) origin = read_origin(st, tick_ps, &errb);
      const uint64_t rel = ticks == 0 ? __builtin_amdgcn_s_memrealtime() : wait_release(origin, ticks);
      if (meas && t == 0) meas[q] = (int64_t)rel;  // release clock; a delay after k_gemv_measured
    });
  }
  if (errb) atomicOr(&st->sticky, errb);
}

__global__ __launch_bounds__(256) void k_gemv_general_timed(const uint16_t *__restrict__ W, int K, int N, int R,
                                                            const uint16_t *__restrict__ X, int B,
                                                            float *__restrict__ Y, int npages,
                                                            const int64_t *__restrict__ pi,
                                                            const int64_t *__restrict__ pc,
                                                            int64_t *__restrict__ meas, int64_t tick_ps,
                                                            DevState *st) {
  timed_pages(npages, pi, pc, meas, tick_ps, st,
              [&](int q, auto wait) { page_general(q, W, K, N, R, X, B, Y, wait); });
}

template <int BB, bool PAD>
__global__ __launch_bounds__(256) void k_gemv_k2048_timed(const uint16_t *__restrict__ W, int N,
                                                          const uint16_t *__restrict__ X, int B_,
                                                          float *__restrict__ Y, int npages,
                                                          const int64_t *__restrict__ pi,
                                                          const int64_t *__restrict__ pc,
                                                          int64_t *__restrict__ meas, int64_t tick_ps,
                                                          DevState *st) {
  __shared__ float red[4][64];
  timed_pages(npages, pi, pc, meas, tick_ps, st,
              [&](int q, auto wait) { page_k2048<BB, PAD>(q, W, N, X, B_, Y, red, wait); });
}

// Persistent grid of a timed kernel: as many workgroups as the GPU holds at
// once, but at least enough that none owns more than GEMV_MAXP pages.
static hipError_t timed_grid(const void *fn, int ncu, int64_t pages, uint32_t *grid) {
  int per_cu = 0;
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, 0);
  if (e != hipSuccess) return e;
  int64_t gsz = (int64_t)(per_cu > 0 ? per_cu : 1) * (ncu > 0 ? ncu : 1);
  if (gsz > pages) gsz = pages;
  const int64_t need = (pages + GEMV_MAXP - 1) / GEMV_MAXP;
  if (gsz < need) gsz = need;
  *grid = (uint32_t)gsz;
  return hipSuccess;
}

static hipError_t finish_measured(int64_t *meas, int64_t pages, int64_t tick_ps, const DevState *st,
                                  hipStream_t s) {
  if (meas)
    hipLaunchKernelGGL(k_gemv_measured, dim3((uint32_t)((pages + 255) / 256)), dim3(256), 0, s, meas, (int)pages,
                       tick_ps, st);
  return hipGetLastError();
}

hipError_t launch_gemv(const uint16_t *W, int E, int K, int N, int page_bytes, const uint16_t *X,
                       int B, float *Y, const int64_t *pi, const int64_t *pc, int64_t *meas,
                       int64_t tick_ps, DevState *st, int ncu, hipStream_t s) {
  const int R = page_bytes / (2 * K);
  const int64_t pages = (int64_t)E * N / R;
  const bool timed = pi != nullptr;
  if (!timed && B >= 9 && B <= 16 && K == 2048 && (N % 32 == 0 || N % 24 == 0)) {
    // 24 rows per workgroup where 32 would leave CUs idle
    if (N % 24 == 0 && ((int64_t)E * N / 32 < ncu || N % 32 != 0))
      hipLaunchKernelGGL(k_gemv_mfma_2t<8>, dim3((uint32_t)((int64_t)E * N / 24)), dim3(512), 0, s, W, N, X, B, Y);
    else
      hipLaunchKernelGGL(k_gemv_mfma_2t<16>, dim3((uint32_t)((int64_t)E * N / 32)), dim3(512), 0, s, W, N, X, B, Y);
    return hipGetLastError();
  }
  if (!timed && B >= 9 && B <= 16 && N % 16 == 0 && K % 512 == 0) {
    const uint32_t tiles = (uint32_t)((int64_t)E * N / 16);
    if (K % 2048 == 0)
      hipLaunchKernelGGL(k_gemv_mfma<16>, dim3(tiles), dim3(256), 0, s, W, K, N, X, B, Y);
    else
      hipLaunchKernelGGL(k_gemv_mfma<4>, dim3(tiles), dim3(256), 0, s, W, K, N, X, B, Y);
    return hipGetLastError();
  }
  if (K == 2048 && R == 4 && B >= 1 && B <= 16) {
    if (!timed) {
      auto kfn = B == 1 ? k_gemv_k2048<1, false> : B == 2 ? k_gemv_k2048<2, false>
               : B == 4 ? k_gemv_k2048<4, false> : B == 8 ? k_gemv_k2048<8, false>
               : B == 16 ? k_gemv_k2048<16, false> : B < 4 ? k_gemv_k2048<4, true>
               : B < 8 ? k_gemv_k2048<8, true> : k_gemv_k2048<16, true>;
      hipLaunchKernelGGL(kfn, dim3((uint32_t)pages), dim3(256), 0, s, W, N, X, B, Y);
      return hipGetLastError();
    }
    auto kfn = B == 1 ? k_gemv_k2048_timed<1, false> : B == 2 ? k_gemv_k2048_timed<2, false>
             : B == 4 ? k_gemv_k2048_timed<4, false> : B == 8 ? k_gemv_k2048_timed<8, false>
             : B == 16 ? k_gemv_k2048_timed<16, false> : B < 4 ? k_gemv_k2048_timed<4, true>
             : B < 8 ? k_gemv_k2048_timed<8, true> : k_gemv_k2048_timed<16, true>;
    uint32_t grid = 0;
    hipError_t e = timed_grid((const void *)kfn, ncu, pages, &grid);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_gemv_origin, dim3(1), dim3(64), 0, s, st);
    hipLaunchKernelGGL(kfn, dim3(grid), dim3(256), 0, s, W, N, X, B, Y, (int)pages, pi, pc, meas, tick_ps, st);
    return finish_measured(meas, pages, tick_ps, st, s);
  }
  if (!timed) {
    hipLaunchKernelGGL(k_gemv_general, dim3((uint32_t)pages), dim3(256), 0, s, W, K, N, R, X, B, Y);
    return hipGetLastError();
  }
  uint32_t grid = 0;
  hipError_t e = timed_grid((const void *)k_gemv_general_timed, ncu, pages, &grid);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_gemv_origin, dim3(1), dim3(64), 0, s, st);
  hipLaunchKernelGGL(k_gemv_general_timed, dim3(grid), dim3(256), 0, s, W, K, N, R, X, B, Y, (int)pages, pi, pc,
                     meas, tick_ps, st);
  return finish_measured(meas, pages, tick_ps, st, s);
}

}  // namespace hbf
