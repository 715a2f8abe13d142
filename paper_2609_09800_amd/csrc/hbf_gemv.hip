// Instrumented bf16 grouped GEMV with HBF delay injection at consumption.
//
// HBFSim (arXiv 2609.09800, Section "D2: Preserving GPU Asynchrony") splits
// an access into issue and consumption: the load is issued and the program
// keeps going; the modeled latency is paid only where the loaded value is
// first used.  Here each workgroup owns one weight page: its waves read the
// wall clock, issue every load of the page, and only then wait -- right
// before the first multiply that consumes the data -- until the page's
// modeled delay has elapsed since the issue.  The wait is measured against
// the GPU's constant-rate wall clock (s_memrealtime); no host clock is
// involved, so no clock origins are mixed.
//
// Y[e][b][n] = sum_k X[e][b][k] * W[e][n][k], bf16 inputs, fp32 accumulate.
// Bandwidth bound (B flop per weight byte): plain FMA, no matrix cores.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbf_internal.h"

namespace hbf {

constexpr int GEMV_MAXV = 8;  // 16-byte weight vectors held per lane
// Longest delay one page may inject; longer requests are clamped to it and
// reported (HBF_ERANGE_TIME) so that a bad time array can never stall the GPU.
constexpr int64_t MAX_PAGE_DELAY_NS = 1000000000;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ float dot8(uint4 w, uint4 x) {
  float s = bf16_lo(w.x) * bf16_lo(x.x);
  s = fmaf(bf16_hi(w.x), bf16_hi(x.x), s);
  s = fmaf(bf16_lo(w.y), bf16_lo(x.y), s);
  s = fmaf(bf16_hi(w.y), bf16_hi(x.y), s);
  s = fmaf(bf16_lo(w.z), bf16_lo(x.z), s);
  s = fmaf(bf16_hi(w.z), bf16_hi(x.z), s);
  s = fmaf(bf16_lo(w.w), bf16_lo(x.w), s);
  s = fmaf(bf16_hi(w.w), bf16_hi(x.w), s);
  return s;
}

// One block (4 wave64) per weight page of R = page_bytes / (2K) rows.
// Wave w takes rows w, w+4, ...; lane l takes the 16-byte vectors
// l, l+64, ... of each row (VPL = K/512 of them).
__global__ __launch_bounds__(256) void k_gemv_instrumented(
    const uint16_t *__restrict__ W, int K, int N, int R, const uint16_t *__restrict__ X, int B,
    float *__restrict__ Y, const int64_t *__restrict__ pi, const int64_t *__restrict__ pc,
    int64_t *__restrict__ meas, int64_t tick_ps, DevState *st) {
  const int q = blockIdx.x;
  const int row0 = q * R;
  const int e = row0 / N;
  const int nb = row0 - e * N;
  const int VPL = K >> 9;
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int RPW = (R + 3) >> 2;

  int64_t d = 0;
  if (pi) {
    d = pc[q] - pi[q];
    if (d < 0) d = 0;
    if (d > MAX_PAGE_DELAY_NS) {
      d = MAX_PAGE_DELAY_NS;
      if (threadIdx.x == 0) atomicOr(&st->sticky, ERR_RANGE_TIME);
    }
  }
  // ceil(d ns / tick), tick in ps
  const uint64_t ticks = (uint64_t)((d * 1000 + tick_ps - 1) / tick_ps);

  // ---- issue: clock, then every load of this page
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
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
  // ---- consumption point: wait for the modeled completion
  uint64_t now = __builtin_amdgcn_s_memrealtime();
  while (now - t0 < ticks) {
    __builtin_amdgcn_s_sleep(1);
    now = __builtin_amdgcn_s_memrealtime();
  }
  if (meas && w == 0 && lane == 0) meas[q] = (int64_t)((now - t0) * (uint64_t)tick_ps / 1000);

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

hipError_t launch_gemv(const uint16_t *W, int E, int K, int N, int page_bytes, const uint16_t *X,
                       int B, float *Y, const int64_t *pi, const int64_t *pc, int64_t *meas,
                       int64_t tick_ps, DevState *st, hipStream_t s) {
  const int R = page_bytes / (2 * K);
  const int64_t pages = (int64_t)E * N / R;
  hipLaunchKernelGGL(k_gemv_instrumented, dim3((uint32_t)pages), dim3(256), 0, s, W, K, N, R, X, B, Y, pi,
                     pc, meas, tick_ps, st);
  return hipGetLastError();
}

}  // namespace hbf
