// Training-step kernels around the sparse backward (App. E): the activity penalties on the
// spike counts of a LIF layer, their gradient added to the layer's spike gradient, and the
// Adam update of a weight matrix.
//
// Penalties, per sample b of a layer with N neurons and counts zeta[b,i] = sum_t S_i[t]:
//   R_low[b] = (lam_low / N) sum_i max(0, nu_low - zeta[b,i])^2
//   R_up[b]  =  lam_up max(0, mean_i zeta[b,i] - nu_up)
// (the appendix prints both with the opposite sign, as terms to maximise; these are the
// penalties minimised), and the loss gains (1/B) sum_b (R_low[b] + R_up[b]). Its derivative
// w.r.t. zeta[b,i], the same for every time step of the neuron, is
//   coef[b,i] = (-2 lam_low / N max(0, nu_low - zeta[b,i]) + [mean_i zeta[b,i] > nu_up] lam_up / N) / B.
//
// HBM: the count reads S once (T B N bytes) plus 4 bytes per (chunk, b, i) of partial counts;
// the gradient add touches 12 bytes per active entry; Adam streams 28 bytes per weight.

#include <algorithm>

#include "common.h"

namespace snn {
namespace {

constexpr int kCountThreads = 256;
constexpr int kCountTargetBlocks = 2048;  // enough blocks to cover the chip several times
constexpr int kRegThreads = 256;
constexpr int kGradRows = 8;  // CSR rows per wave in the gradient add

struct CountPlan {
  int chunks, chunk_len;
  int64_t BN;
};

CountPlan count_plan(int T, int B, int N) {
  CountPlan p;
  p.BN = (int64_t)B * N;
  const int64_t quads = (p.BN + 3) / 4;
  const int64_t bx = (quads + kCountThreads - 1) / kCountThreads;
  int want = (int)std::min<int64_t>((kCountTargetBlocks + bx - 1) / bx, T);
  want = std::max(want, 1);
  p.chunk_len = (T + want - 1) / want;
  p.chunks = (T + p.chunk_len - 1) / p.chunk_len;
  return p;
}

// Partial spike counts over steps [c*chunk_len, min(T, (c+1)*chunk_len)) of chunk c = blockIdx.y.
// VEC: each thread counts 4 neighbouring bytes of a [T][B*N] row with one 32-bit load per step
// (B*N a multiple of 4 and S 4-byte aligned); else one byte per thread.
template <bool VEC>
__global__ void __launch_bounds__(kCountThreads) count_chunks(const uint8_t* __restrict__ S, int T, int64_t BN,
                                                              int chunk_len, int32_t* __restrict__ partial) {
  const int c = blockIdx.y;
  const int t0 = c * chunk_len;
  const int t1 = min(T, t0 + chunk_len);
  const int64_t q = (int64_t)blockIdx.x * kCountThreads + threadIdx.x;
  int32_t* out = partial + (int64_t)c * BN;
  if (VEC) {
    const int64_t k = q * 4;
    if (k >= BN) return;
    int n0 = 0, n1 = 0, n2 = 0, n3 = 0;
#pragma unroll 8
    for (int t = t0; t < t1; ++t) {
      const uint32_t x = *reinterpret_cast<const uint32_t*>(S + (int64_t)t * BN + k);
      n0 += (x & 0xffu) != 0u;
      n1 += (x & 0xff00u) != 0u;
      n2 += (x & 0xff0000u) != 0u;
      n3 += (x & 0xff000000u) != 0u;
    }
    *reinterpret_cast<int4*>(out + k) = make_int4(n0, n1, n2, n3);
  } else {
    if (q >= BN) return;
    int n = 0;
#pragma unroll 8
    for (int t = t0; t < t1; ++t) n += S[(int64_t)t * BN + q] != 0;
    out[q] = n;
  }
}

__device__ __forceinline__ double block_sum(double v, double* red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  for (int s = kRegThreads / 2; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__device__ __forceinline__ int count_of(const int32_t* __restrict__ partial, int chunks, int64_t BN, int64_t k) {
  int z = 0;
  for (int c = 0; c < chunks; ++c) z += partial[(int64_t)c * BN + k];
  return z;
}

// One block per sample b: counts, the per-sample penalty and the coefficient of every neuron.
// Sums run in float64 in a fixed order, so the results are deterministic.
__global__ void __launch_bounds__(kRegThreads) reg_sample(const int32_t* __restrict__ partial, int chunks, int B,
                                                          int N, float lam_low, float nu_low, float lam_up,
                                                          float nu_up, int32_t* __restrict__ zeta,
                                                          float* __restrict__ coef, double* __restrict__ pen_b) {
  __shared__ double red[kRegThreads];
  const int b = blockIdx.x;
  const int64_t BN = (int64_t)B * N;
  const int64_t row = (int64_t)b * N;
  double s_z = 0.0, s_low = 0.0;
  for (int i = threadIdx.x; i < N; i += kRegThreads) {
    const int z = count_of(partial, chunks, BN, row + i);
    if (zeta) zeta[row + i] = z;
    s_z += (double)z;
    const double d = fmax(0.0, (double)nu_low - (double)z);
    s_low += d * d;
  }
  s_z = block_sum(s_z, red);
  s_low = block_sum(s_low, red);
  const double mean = s_z / (double)N;
  const bool up = mean > (double)nu_up;
  if (threadIdx.x == 0) pen_b[b] = (double)lam_low / (double)N * s_low + (double)lam_up * fmax(0.0, mean - (double)nu_up);
  const double inv_b = 1.0 / (double)B;
  const double c_up = up ? (double)lam_up / (double)N : 0.0;
  const double c_low = -2.0 * (double)lam_low / (double)N;
  for (int i = threadIdx.x; i < N; i += kRegThreads) {
    const int z = count_of(partial, chunks, BN, row + i);
    coef[row + i] = (float)((c_low * fmax(0.0, (double)nu_low - (double)z) + c_up) * inv_b);
  }
}

// penalty = (1/B) sum_b pen_b[b], one block, fixed order.
__global__ void __launch_bounds__(kRegThreads) reg_mean(const double* __restrict__ pen_b, int B,
                                                        float* __restrict__ penalty) {
  __shared__ double red[kRegThreads];
  double s = 0.0;
  for (int b = threadIdx.x; b < B; b += kRegThreads) s += pen_b[b];
  s = block_sum(s, red);
  if (threadIdx.x == 0) *penalty = (float)(s / (double)B);
}

// eps[e] += coef[b(e), col(e)] over the CSR entries; each wave takes kGradRows rows, whose entries
// are contiguous, and finds the row of an entry by comparing with the row starts it holds.
// Entries are clamped to [0, capacity) and columns outside [0, N) are skipped.
__global__ void __launch_bounds__(256) reg_grad_csr(const float* __restrict__ coef, int TB, int B, int N,
                                                    const int32_t* __restrict__ row_ptr,
                                                    const int32_t* __restrict__ col_idx, int64_t capacity,
                                                    float* __restrict__ eps) {
  const int wave = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
  const int r0 = wave * kGradRows;
  if (r0 >= TB) return;
  const int nr = min(kGradRows, TB - r0);
  int starts[kGradRows + 1];
#pragma unroll
  for (int k = 0; k <= kGradRows; ++k) starts[k] = row_ptr[r0 + min(k, nr)];
  const int64_t lo = max(0, starts[0]);
  const int64_t hi = min((int64_t)starts[nr], capacity);
  for (int64_t e = lo + lane_id(); e < hi; e += kWave) {
    int k = 0;
#pragma unroll
    for (int j = 1; j < kGradRows; ++j) k += (j < nr && e >= starts[j]) ? 1 : 0;
    const int b = (r0 + k) % B;
    const int col = col_idx[e];
    if ((unsigned)col < (unsigned)N) eps[e] += coef[(int64_t)b * N + col];
  }
}

// Dense form: eps[t,b,i] += coef[b,i].
template <bool VEC>
__global__ void __launch_bounds__(256) reg_grad_dense(const float* __restrict__ coef, int64_t total, int64_t BN,
                                                      float* __restrict__ eps) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (VEC) {
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q * 4 < total; q += stride) {
      const int64_t e = q * 4;
      const int64_t k = e % BN;  // BN % 4 == 0, so the four entries share t
      float4 x = *reinterpret_cast<float4*>(eps + e);
      const float4 c = *reinterpret_cast<const float4*>(coef + k);
      x.x += c.x;
      x.y += c.y;
      x.z += c.z;
      x.w += c.w;
      *reinterpret_cast<float4*>(eps + e) = x;
    }
  } else {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += stride) eps[e] += coef[e % BN];
  }
}

// Adam (Kingma and Ba, Algorithm 1) in float32:
//   m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;  w -= step_size * m / (sqrt(v) * rs + eps)
// with step_size = lr / (1 - b1^k) and rs = 1 / sqrt(1 - b2^k) formed on the host in float64.
struct AdamArgs {
  float b1, one_m_b1, b2, one_m_b2, eps, step_size, rs;
};

__device__ __forceinline__ void adam_one(float& w, float g, float& m, float& v, const AdamArgs& a) {
  m = a.b1 * m + a.one_m_b1 * g;
  v = a.b2 * v + a.one_m_b2 * (g * g);
  w -= a.step_size * (m / (sqrtf(v) * a.rs + a.eps));
}

template <bool VEC>
__global__ void __launch_bounds__(256) adam_kernel(float* __restrict__ W, const float* __restrict__ grad,
                                                   float* __restrict__ m, float* __restrict__ v, int64_t n,
                                                   AdamArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (VEC) {
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q * 4 < n; q += stride) {
      float4 w = reinterpret_cast<float4*>(W)[q];
      const float4 g = reinterpret_cast<const float4*>(grad)[q];
      float4 mm = reinterpret_cast<float4*>(m)[q];
      float4 vv = reinterpret_cast<float4*>(v)[q];
      adam_one(w.x, g.x, mm.x, vv.x, a);
      adam_one(w.y, g.y, mm.y, vv.y, a);
      adam_one(w.z, g.z, mm.z, vv.z, a);
      adam_one(w.w, g.w, mm.w, vv.w, a);
      reinterpret_cast<float4*>(W)[q] = w;
      reinterpret_cast<float4*>(m)[q] = mm;
      reinterpret_cast<float4*>(v)[q] = vv;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
      float w = W[i], mm = m[i], vv = v[i];
      adam_one(w, grad[i], mm, vv, a);
      W[i] = w;
      m[i] = mm;
      v[i] = vv;
    }
  }
}

inline bool finite_nonneg(float x) { return x >= 0.0f && x <= 3.4e38f; }  // rejects NaN and inf
inline bool finite(float x) { return x >= -3.4e38f && x <= 3.4e38f; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

unsigned stream_blocks(int64_t items) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 8192));
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" size_t snn_activity_reg_workspace(int T, int B, int N) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return 0;
  const CountPlan p = count_plan(T, B, N);
  Carve c(nullptr);
  c.take<int32_t>((size_t)p.chunks * (size_t)p.BN);
  c.take<double>((size_t)B);
  return c.off;
}

extern "C" snn_status snn_activity_reg(const uint8_t* S, int T, int B, int N, float lam_low, float nu_low,
                                       float lam_up, float nu_up, int32_t* zeta, float* coef, float* penalty,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  if (!S || !coef || !workspace) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return SNN_ERR_INVALID_ARG;
  if (!finite_nonneg(lam_low) || !finite_nonneg(lam_up) || !finite(nu_low) || !finite(nu_up))
    return SNN_ERR_INVALID_ARG;
  if (workspace_bytes < snn_activity_reg_workspace(T, B, N)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const CountPlan p = count_plan(T, B, N);
  Carve ws(workspace);
  int32_t* partial = ws.take<int32_t>((size_t)p.chunks * (size_t)p.BN);
  double* pen_b = ws.take<double>((size_t)B);
  const bool vec = (p.BN % 4 == 0) && (((uintptr_t)S & 3u) == 0);
  if (vec) {
    const int64_t quads = p.BN / 4;
    dim3 grid((unsigned)((quads + kCountThreads - 1) / kCountThreads), (unsigned)p.chunks);
    hipLaunchKernelGGL(count_chunks<true>, grid, dim3(kCountThreads), 0, s, S, T, p.BN, p.chunk_len, partial);
  } else {
    dim3 grid((unsigned)((p.BN + kCountThreads - 1) / kCountThreads), (unsigned)p.chunks);
    hipLaunchKernelGGL(count_chunks<false>, grid, dim3(kCountThreads), 0, s, S, T, p.BN, p.chunk_len, partial);
  }
  hipLaunchKernelGGL(reg_sample, dim3(B), dim3(kRegThreads), 0, s, partial, p.chunks, B, N, lam_low, nu_low, lam_up,
                     nu_up, zeta, coef, pen_b);
  if (penalty) hipLaunchKernelGGL(reg_mean, dim3(1), dim3(kRegThreads), 0, s, pen_b, B, penalty);
  return launch_status();
}

extern "C" snn_status snn_activity_reg_grad(const float* coef, int T, int B, int N, const int32_t* row_ptr,
                                            const int32_t* col_idx, int64_t capacity, float* eps, void* stream) {
  if (!coef || !eps) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (row_ptr) {
    if (!col_idx || capacity < 0) return SNN_ERR_INVALID_ARG;
    const int TB = T * B;
    const int64_t waves = (TB + kGradRows - 1) / kGradRows;
    const unsigned blocks = (unsigned)((waves * kWave + 255) / 256);
    if (capacity > 0)
      hipLaunchKernelGGL(reg_grad_csr, dim3(blocks), dim3(256), 0, s, coef, TB, B, N, row_ptr, col_idx, capacity, eps);
  } else {
    const int64_t BN = (int64_t)B * N;
    const int64_t total = BN * T;
    if (BN % 4 == 0 && aligned16(eps) && aligned16(coef))
      hipLaunchKernelGGL(reg_grad_dense<true>, dim3(stream_blocks(total / 4)), dim3(256), 0, s, coef, total, BN, eps);
    else
      hipLaunchKernelGGL(reg_grad_dense<false>, dim3(stream_blocks(total)), dim3(256), 0, s, coef, total, BN, eps);
  }
  return launch_status();
}

extern "C" snn_status snn_adam_step(float* W, const float* grad, float* m, float* v, int64_t n, float lr,
                                    float beta1, float beta2, float eps, int step, void* stream) {
  if (!W || !grad || !m || !v || n <= 0 || step < 1) return SNN_ERR_INVALID_ARG;
  if (!finite_nonneg(lr) || !(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f) ||
      !(eps > 0.0f && eps <= 3.4e38f))
    return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  AdamArgs a;
  a.b1 = beta1;
  a.one_m_b1 = (float)(1.0 - (double)beta1);
  a.b2 = beta2;
  a.one_m_b2 = (float)(1.0 - (double)beta2);
  a.eps = eps;
  a.step_size = (float)((double)lr / (1.0 - pow((double)beta1, (double)step)));
  a.rs = (float)(1.0 / sqrt(1.0 - pow((double)beta2, (double)step)));
  const bool vec = n % 4 == 0 && aligned16(W) && aligned16(grad) && aligned16(m) && aligned16(v);
  if (vec)
    hipLaunchKernelGGL(adam_kernel<true>, dim3(stream_blocks(n / 4)), dim3(256), 0, s, W, grad, m, v, n, a);
  else
    hipLaunchKernelGGL(adam_kernel<false>, dim3(stream_blocks(n)), dim3(256), 0, s, W, grad, m, v, n, a);
  return launch_status();
}
