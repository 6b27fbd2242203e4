// LIF forward of one fully connected layer (Sec. 2.1): Eq. (lif) with V_rest = V_r = 0,
// V[0] = 0, the strict Heaviside of Eq. (spike_fn), and the input trace that Eq. (w_grad)
// reuses (the filtered input of Eq. (lif_unrolled)).
//
// One block owns one batch sample b and up to 256 output neurons j (one per thread); the
// j-blocks of a sample are placed on the same XCD so they share its L2 for the spike rows.
// Time is walked in chunks of P steps:
//   1. each wavefront turns some of the chunk's spike rows S_in[t,b,:] into an ascending list
//      of spiking inputs in LDS (wave ballot per byte lane + mbcnt prefix);
//   2. every thread sums W[i,j] over each list in ascending i for all P rows at once (the P
//      independent gathers keep many W loads in flight; W rows are served by L2);
//   3. the membrane recurrence runs P steps in registers and writes V and S_out;
//   4. the block updates its share of the input trace and writes it.
// Float32 with separately rounded operations (__fmul_rn / __fadd_rn) and the ascending
// summation order make V a deterministic function of the inputs.
#include "common.h"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int kJT = 256;         // output neurons per block
constexpr int kPMax = 16;        // time steps per chunk
constexpr int kTraceGroups = 4;  // float4 trace groups per thread -> 4096 inputs per block
constexpr int kListBytes = 32768;

template <bool ALIGNED>
__device__ __forceinline__ uint32_t load4(const uint8_t* p, int i, int n) {
  if (ALIGNED) return i < n ? *reinterpret_cast<const uint32_t*>(p + i) : 0u;
  uint32_t x = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (i + q < n) x |= (uint32_t)p[i + q] << (8 * q);
  return x;
}

template <bool ALIGNED>
__global__ __launch_bounds__(kThreads) void lif_forward_kernel(const uint8_t* __restrict__ s_in,
                                                               const float* __restrict__ W, int T, int B, int N_in,
                                                               int N_out, float alpha, float theta,
                                                               float* __restrict__ V, uint8_t* __restrict__ s_out,
                                                               float* __restrict__ trace, int P, int n_jblk,
                                                               int tr_span) {
  extern __shared__ uint16_t lists[];  // [P][N_in]
  __shared__ int counts[kPMax];

  int id = blockIdx.x;
  const int G = gridDim.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);  // consecutive ids share an XCD
  const int b = id / n_jblk;
  const int jb = id - b * n_jblk;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int j = jb * kJT + tid;
  const bool has_j = j < N_out;

  const size_t step_in = (size_t)B * N_in;
  const size_t step_out = (size_t)B * N_out;
  const int tr_lo = jb * tr_span;
  const int tr_hi = min(N_in, tr_lo + tr_span);
  float tr[kTraceGroups][4];
#pragma unroll
  for (int k = 0; k < kTraceGroups; ++k)
#pragma unroll
    for (int q = 0; q < 4; ++q) tr[k][q] = 0.0f;

  float v = 0.0f;
  if (has_j) V[(size_t)b * N_out + j] = 0.0f;
  if (trace) {
#pragma unroll
    for (int k = 0; k < kTraceGroups; ++k) {
      const int i = tr_lo + 4 * (tid + kThreads * k);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (i + q < tr_hi) trace[(size_t)b * N_in + i + q] = 0.0f;
    }
  }

  for (int t0 = 0; t0 < T - 1; t0 += P) {
    const int np = min(P, T - 1 - t0);
    // 1. ascending lists of spiking inputs, one row per wavefront at a time
    for (int p = w; p < np; p += kThreads / kWave) {
      const uint8_t* row = s_in + (size_t)(t0 + p) * step_in + (size_t)b * N_in;
      uint16_t* lst = lists + p * N_in;
      int base = 0;
      for (int i0 = 0; i0 < N_in; i0 += 4 * kWave) {
        const int i = i0 + 4 * l;
        const uint32_t x = load4<ALIGNED>(row, i, N_in);
        const bool a0 = (x & 0xffu) != 0, a1 = (x & 0xff00u) != 0, a2 = (x & 0xff0000u) != 0,
                   a3 = (x & 0xff000000u) != 0;
        const uint64_t m0 = __ballot(a0), m1 = __ballot(a1), m2 = __ballot(a2), m3 = __ballot(a3);
        int pos = base + mask_prefix(m0) + mask_prefix(m1) + mask_prefix(m2) + mask_prefix(m3);
        if (a0) lst[pos++] = (uint16_t)i;
        if (a1) lst[pos++] = (uint16_t)(i + 1);
        if (a2) lst[pos++] = (uint16_t)(i + 2);
        if (a3) lst[pos++] = (uint16_t)(i + 3);
        base += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
      }
      if (l == 0) counts[p] = base;
    }
    __syncthreads();

    // 2-3. weighted inputs of the chunk, then the membrane recurrence
    if (has_j) {
      float acc[kPMax];
      int cnt[kPMax];
      int kmax = 0;
#pragma unroll
      for (int p = 0; p < kPMax; ++p) {
        acc[p] = 0.0f;
        cnt[p] = p < np ? counts[p] : 0;
        kmax = max(kmax, cnt[p]);
      }
      const float* Wj = W + j;
      for (int k = 0; k < kmax; ++k) {
#pragma unroll
        for (int p = 0; p < kPMax; ++p)
          if (k < cnt[p]) acc[p] = __fadd_rn(acc[p], Wj[(size_t)lists[p * N_in + k] * N_out]);
      }
#pragma unroll
      for (int p = 0; p < kPMax; ++p) {
        if (p < np) {
          const int t = t0 + p;
          const bool s = v > theta;
          s_out[(size_t)t * step_out + (size_t)b * N_out + j] = (uint8_t)s;
          v = __fadd_rn(__fadd_rn(__fmul_rn(alpha, v), acc[p]), s ? -1.0f : -0.0f);
          V[(size_t)(t + 1) * step_out + (size_t)b * N_out + j] = v;
        }
      }
    }

    // 4. input trace of this block's share of the inputs
    if (trace) {
#pragma unroll
      for (int k = 0; k < kTraceGroups; ++k) {
        const int i = tr_lo + 4 * (tid + kThreads * k);
        if (i < tr_hi) {
          for (int p = 0; p < np; ++p) {
            const uint32_t x = load4<ALIGNED>(s_in + (size_t)(t0 + p) * step_in + (size_t)b * N_in, i, N_in);
#pragma unroll
            for (int q = 0; q < 4; ++q)
              tr[k][q] = __fadd_rn(__fmul_rn(alpha, tr[k][q]), ((x >> (8 * q)) & 0xffu) ? 1.0f : 0.0f);
            float* dst = trace + (size_t)(t0 + p + 1) * step_in + (size_t)b * N_in + i;
            if (ALIGNED && i + 3 < tr_hi) {
              *reinterpret_cast<float4*>(dst) = make_float4(tr[k][0], tr[k][1], tr[k][2], tr[k][3]);
            } else {
#pragma unroll
              for (int q = 0; q < 4; ++q)
                if (i + q < tr_hi) dst[q] = tr[k][q];
            }
          }
        }
      }
    }
    __syncthreads();
  }
  if (has_j) s_out[(size_t)(T - 1) * step_out + (size_t)b * N_out + j] = (uint8_t)(v > theta);
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" snn_status snn_lif_forward(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                      float alpha, float theta, float* V, uint8_t* s_out, float* trace_in,
                                      void* stream) {
  if (!s_in || !W || !V || !s_out) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || isnan(theta)) return SNN_ERR_INVALID_ARG;
  if (N_in > kTraceGroups * kThreads * 4) return SNN_ERR_UNSUPPORTED;

  const int n_jblk = (N_out + kJT - 1) / kJT;
  int tr_span = (N_in + n_jblk - 1) / n_jblk;
  tr_span = (tr_span + 3) & ~3;
  const int P = max(1, min(kPMax, kListBytes / (int)(N_in * sizeof(uint16_t))));
  const size_t lds = (size_t)P * N_in * sizeof(uint16_t);
  const bool aligned = (N_in % 4) == 0 && (reinterpret_cast<uintptr_t>(s_in) % 4) == 0 &&
                       (reinterpret_cast<uintptr_t>(trace_in) % 16) == 0;
  const dim3 grid((unsigned)B * n_jblk);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (aligned)
    hipLaunchKernelGGL(lif_forward_kernel<true>, grid, dim3(kThreads), lds, s, s_in, W, T, B, N_in, N_out, alpha,
                       theta, V, s_out, trace_in, P, n_jblk, tr_span);
  else
    hipLaunchKernelGGL(lif_forward_kernel<false>, grid, dim3(kThreads), lds, s, s_in, W, T, B, N_in, N_out, alpha,
                       theta, V, s_out, trace_in, P, n_jblk, tr_span);
  return launch_status();
}
