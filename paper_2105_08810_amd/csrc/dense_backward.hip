// Dense surrogate BPTT of one layer -- the "Original" column of Table 1 -- on fp32 matrix cores.
//
//   gate+delta  one thread per (b,j) walks t downward: G = eps * g(V) * 1[band] (or eps for the
//               readout), delta[t-1] = alpha delta[t] + G[t]; writes G and delta densely.
//   grad_in     [T*B, N_in] = delta [T*B, N_out] . W^T      (GEMM, both operands K-contiguous)
//   dW          [N_in, N_out] = trace^T [N_in, T*B] . G     (GEMM, K = T*B, split over K)
// The GEMM is a 128x128x16 tile per 256-thread block; each wavefront owns 64x64 as 2x2
// v_mfma_f32_32x32x2f32 accumulators, operands staged through LDS (k-major, padded).
#include "common.h"

namespace snn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 16, PAD = 4;
constexpr int kGemmThreads = 256;

__device__ __forceinline__ float gate(float e, float v, float theta, float bth, float beta, bool readout) {
  if (readout) return e;
  const float d = fabsf(v - theta);
  if (!(d < bth)) return 0.0f;
  const float x = beta * d + 1.0f;
  return e / (x * x);
}

__global__ __launch_bounds__(256) void dense_gate_delta(const float* __restrict__ eps, const float* __restrict__ V,
                                                        int T, size_t BN_, float alpha, float theta, float bth,
                                                        float beta, int readout, float* __restrict__ Gd,
                                                        float* __restrict__ Dd) {
  const size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (k >= BN_) return;
  const bool ro = readout != 0;
  float d = 0.0f;
  Dd[(size_t)(T - 1) * BN_ + k] = 0.0f;
  constexpr int U = 4;
  int t = T - 1;
  for (; t >= U - 1; t -= U) {  // independent loads of U steps in flight
    float e[U], v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t o = (size_t)(t - u) * BN_ + k;
      e[u] = eps[o];
      v[u] = ro ? 0.0f : V[o];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tt = t - u;
      const float G = gate(e[u], v[u], theta, bth, beta, ro);
      Gd[(size_t)tt * BN_ + k] = G;
      if (tt > 0) {
        d = alpha * d + G;
        Dd[(size_t)(tt - 1) * BN_ + k] = d;
      }
    }
  }
  for (; t >= 0; --t) {
    const size_t o = (size_t)t * BN_ + k;
    const float G = gate(eps[o], ro ? 0.0f : V[o], theta, bth, beta, ro);
    Gd[o] = G;
    if (t > 0) {
      d = alpha * d + G;
      Dd[(size_t)(t - 1) * BN_ + k] = d;
    }
  }
}

// C[M x N] = sum_k A(m,k) B(k,n) over this block's K slice.
//   A_KM: A(m,k) = A[k*lda + m] (m contiguous)   else A[m*lda + k] (k contiguous)
//   B_KN: B(k,n) = B[k*ldb + n] (n contiguous)   else B[n*ldb + k] (k contiguous)
// Block z = K slice; its output goes to C + z * c_split.
template <bool A_KM, bool B_KN, bool VEC>
__global__ __launch_bounds__(kGemmThreads) void gemm_f32_mfma(int M, int N, int K, const float* __restrict__ A,
                                                              int lda, const float* __restrict__ B, int ldb,
                                                              float* __restrict__ C, int ldc, int k_per_split,
                                                              size_t c_split, int tiles_n) {
  __shared__ float As[2][BK][BM + PAD];
  __shared__ float Bs[2][BK][BN + PAD];
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int tm = blockIdx.x / tiles_n;
  const int tn = blockIdx.x - tm * tiles_n;
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int k_lo = blockIdx.y * k_per_split;
  const int k_hi = min(K, k_lo + k_per_split);
  const int wm = (w / 2) * 64;
  const int wn = (w % 2) * 64;

  floatx16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  // register staging of one K tile: 2 float4 per thread per operand
  float ra[2][4], rb[2][4];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + kGemmThreads * q;
      if (A_KM) {  // tile [BK][BM]: kk = idx/32, m4 = idx%32
        const int kk = idx / 32, mm = 4 * (idx % 32);
        const int kg = k0 + kk, mg = m0 + mm;
        if (VEC && kg < k_hi && mg + 3 < M) {
          const float4 v = *reinterpret_cast<const float4*>(A + (size_t)kg * lda + mg);
          ra[q][0] = v.x; ra[q][1] = v.y; ra[q][2] = v.z; ra[q][3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) ra[q][c] = (kg < k_hi && mg + c < M) ? A[(size_t)kg * lda + mg + c] : 0.0f;
        }
      } else {  // tile [BM][BK]: mm = idx/4, k4 = idx%4
        const int mm = idx / 4, kk = 4 * (idx % 4);
        const int kg = k0 + kk, mg = m0 + mm;
        if (VEC && mg < M && kg + 3 < k_hi) {
          const float4 v = *reinterpret_cast<const float4*>(A + (size_t)mg * lda + kg);
          ra[q][0] = v.x; ra[q][1] = v.y; ra[q][2] = v.z; ra[q][3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) ra[q][c] = (mg < M && kg + c < k_hi) ? A[(size_t)mg * lda + kg + c] : 0.0f;
        }
      }
      if (B_KN) {
        const int kk = idx / 32, nn = 4 * (idx % 32);
        const int kg = k0 + kk, ng = n0 + nn;
        if (VEC && kg < k_hi && ng + 3 < N) {
          const float4 v = *reinterpret_cast<const float4*>(B + (size_t)kg * ldb + ng);
          rb[q][0] = v.x; rb[q][1] = v.y; rb[q][2] = v.z; rb[q][3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) rb[q][c] = (kg < k_hi && ng + c < N) ? B[(size_t)kg * ldb + ng + c] : 0.0f;
        }
      } else {
        const int nn = idx / 4, kk = 4 * (idx % 4);
        const int kg = k0 + kk, ng = n0 + nn;
        if (VEC && ng < N && kg + 3 < k_hi) {
          const float4 v = *reinterpret_cast<const float4*>(B + (size_t)ng * ldb + kg);
          rb[q][0] = v.x; rb[q][1] = v.y; rb[q][2] = v.z; rb[q][3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) rb[q][c] = (ng < N && kg + c < k_hi) ? B[(size_t)ng * ldb + kg + c] : 0.0f;
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + kGemmThreads * q;
      if (A_KM) {
        const int kk = idx / 32, mm = 4 * (idx % 32);
        *reinterpret_cast<float4*>(&As[buf][kk][mm]) = make_float4(ra[q][0], ra[q][1], ra[q][2], ra[q][3]);
      } else {
        const int mm = idx / 4, kk = 4 * (idx % 4);
#pragma unroll
        for (int c = 0; c < 4; ++c) As[buf][kk + c][mm] = ra[q][c];
      }
      if (B_KN) {
        const int kk = idx / 32, nn = 4 * (idx % 32);
        *reinterpret_cast<float4*>(&Bs[buf][kk][nn]) = make_float4(rb[q][0], rb[q][1], rb[q][2], rb[q][3]);
      } else {
        const int nn = idx / 4, kk = 4 * (idx % 4);
#pragma unroll
        for (int c = 0; c < 4; ++c) Bs[buf][kk + c][nn] = rb[q][c];
      }
    }
  };

  const int ntiles = (k_hi - k_lo + BK - 1) / BK;
  if (ntiles > 0) {
    load_tile(k_lo);
    store_tile(0);
  }
  __syncthreads();
  const int lr = l % 32;
  const int lk = l / 32;
  for (int kt = 0; kt < ntiles; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < ntiles) load_tile(k_lo + (kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      const float a0 = As[cur][kk + lk][wm + lr];
      const float a1 = As[cur][kk + lk][wm + 32 + lr];
      const float b0 = Bs[cur][kk + lk][wn + lr];
      const float b1 = Bs[cur][kk + lk][wn + 32 + lr];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    if (kt + 1 < ntiles) store_tile(cur ^ 1);
    __syncthreads();
  }

  // accumulator layout of 32x32x2: register v of lane l holds row 8*(v/4) + 4*(l/32) + v%4, column l%32
  float* Cz = C + (size_t)blockIdx.y * c_split;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm + 32 * a + 8 * (v / 4) + 4 * lk + (v % 4);
        const int n = n0 + wn + 32 * b + lr;
        if (m < M && n < N) Cz[(size_t)m * ldc + n] = acc[a][b][v];
      }
}

__global__ void reduce_splits(const float* __restrict__ part, int n_split, size_t n, float* __restrict__ out) {
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    double s = 0.0;  // fixed order, rounded once
    for (int c = 0; c < n_split; ++c) s += (double)part[(size_t)c * n + k];
    out[k] = (float)s;
  }
}

int dw_splits(int TB, int N_in, int N_out) {
  const int tiles = ((N_in + BM - 1) / BM) * ((N_out + BN - 1) / BN);
  int s = (2 * cu_count() + tiles - 1) / tiles;
  s = std::min(s, std::max(1, TB / 256));
  return std::max(1, std::min(s, 64));
}

template <bool A_KM, bool B_KN>
void launch_gemm(bool vec, int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C, int ldc,
                 int splits, size_t c_split, hipStream_t s) {
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  int kps = (K + splits - 1) / splits;
  kps = (kps + BK - 1) / BK * BK;
  const dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)splits);
  if (vec)
    hipLaunchKernelGGL((gemm_f32_mfma<A_KM, B_KN, true>), grid, dim3(kGemmThreads), 0, s, M, N, K, A, lda, B, ldb, C,
                       ldc, kps, c_split, tiles_n);
  else
    hipLaunchKernelGGL((gemm_f32_mfma<A_KM, B_KN, false>), grid, dim3(kGemmThreads), 0, s, M, N, K, A, lda, B, ldb,
                       C, ldc, kps, c_split, tiles_n);
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" size_t snn_dense_backward_workspace(int T, int B, int N_in, int N_out) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return 0;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return 0;
  const size_t TB = (size_t)T * B;
  Carve c(nullptr);
  c.take<float>(TB * N_out);  // G
  c.take<float>(TB * N_out);  // delta
  const int sp = dw_splits(T * B, N_in, N_out);
  if (sp > 1) c.take<float>((size_t)sp * N_in * N_out);
  return c.off;
}

extern "C" snn_status snn_dense_backward_ref(const float* W, const float* trace_in, const float* V,
                                             const float* eps_out, int T, int B, int N_in, int N_out, float alpha,
                                             float theta, float b_th, float beta, float* grad_in, float* dW,
                                             void* workspace, size_t workspace_bytes, void* stream) {
  if (!W || !trace_in || !eps_out || !dW || !workspace) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || isnan(theta) || isnan(b_th) || b_th < 0.0f || isnan(beta) || beta < 0.0f)
    return SNN_ERR_INVALID_ARG;
  const bool readout = isinf(theta) && theta > 0.0f;
  if (!readout && !V) return SNN_ERR_INVALID_ARG;
  if (workspace_bytes < snn_dense_backward_workspace(T, B, N_in, N_out)) return SNN_ERR_INVALID_ARG;

  hipStream_t s = static_cast<hipStream_t>(stream);
  const int TB = T * B;
  Carve ws(workspace);
  float* Gd = ws.take<float>((size_t)TB * N_out);
  float* Dd = ws.take<float>((size_t)TB * N_out);
  const int sp = dw_splits(TB, N_in, N_out);
  float* part = sp > 1 ? ws.take<float>((size_t)sp * N_in * N_out) : dW;

  const size_t BN_ = (size_t)B * N_out;
  hipLaunchKernelGGL(dense_gate_delta, dim3((unsigned)((BN_ + 255) / 256)), dim3(256), 0, s, eps_out, V, T, BN_,
                     alpha, theta, b_th, beta, readout ? 1 : 0, Gd, Dd);
  const bool vec_dw = (N_in % 4 == 0) && (N_out % 4 == 0);
  // dW[i][j] = sum_r trace[r][i] G[r][j]: A(m=i,k=r) = trace[r*N_in + i], B(k=r,n=j) = G[r*N_out + j]
  launch_gemm<true, true>(vec_dw, N_in, N_out, TB, trace_in, N_in, Gd, N_out, part, N_out, sp,
                          (size_t)N_in * N_out, s);
  if (sp > 1) {
    const size_t n = (size_t)N_in * N_out;
    hipLaunchKernelGGL(reduce_splits, dim3((unsigned)std::min<size_t>((n + 255) / 256, 4096)), dim3(256), 0, s,
                       part, sp, n, dW);
  }
  if (grad_in) {
    // grad_in[r][i] = sum_j delta[r][j] W[i][j]: A(m=r,k=j) = delta[r*N_out + j], B(k=j,n=i) = W[i*N_out + j]
    const bool vec_gi = (N_out % 4 == 0);
    launch_gemm<false, false>(vec_gi, TB, N_in, N_out, Dd, N_out, W, N_out, grad_in, N_in, 1, 0, s);
  }
  return launch_status();
}
