// Readout cross-entropy (App. E) and the CSR of the entries the loss reads, so that the
// readout's backward runs through snn_sparse_backward like any other layer. The readout is
// the infinite-threshold LIF layer of Sec. 3; its derivative factor is 1.
//   mode 0: a[b,c] = max_t V_out[t,b,c] (first maximal t), entries = the arg-max positions
//   mode 1: a[b,c] = sum_t V_out[t,b,c], entries = every (t,b,c)
// eps = dL/da = (softmax(a) - onehot(label)) / B at each entry; loss = mean -log p[b,label].
#include "common.h"

namespace snn {
namespace {

constexpr int kThreads = 256;

// One block per sample b: logits, softmax, per-sample loss, dL/da and arg-max times.
__global__ __launch_bounds__(kThreads) void ce_sample(const float* __restrict__ V, const int32_t* __restrict__ labels,
                                                      int T, int B, int C, int mode, int32_t* __restrict__ tstar,
                                                      float* __restrict__ dlda, float* __restrict__ loss_b) {
  extern __shared__ float a[];  // [C]
  __shared__ float red[kThreads / kWave];
  __shared__ float bc[2];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  for (int c = tid; c < C; c += kThreads) {
    if (mode == 0) {
      float best = V[(size_t)b * C + c];
      int bt = 0;
      for (int t = 1; t < T; ++t) {
        const float v = V[((size_t)t * B + b) * C + c];
        if (v > best) {
          best = v;
          bt = t;
        }
      }
      a[c] = best;
      tstar[(size_t)b * C + c] = bt;
    } else {
      double s = 0.0;  // the logit of a sum over time, rounded once
      for (int t = 0; t < T; ++t) s += (double)V[((size_t)t * B + b) * C + c];
      a[c] = (float)s;
    }
  }
  __syncthreads();
  // max over classes
  float m = -INFINITY;
  for (int c = tid; c < C; c += kThreads) m = fmaxf(m, a[c]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
  if (l == 0) red[w] = m;
  __syncthreads();
  if (tid == 0) {
    float mm = red[0];
    for (int k = 1; k < kThreads / kWave; ++k) mm = fmaxf(mm, red[k]);
    bc[0] = mm;
  }
  __syncthreads();
  const float amax = bc[0];
  float s = 0.0f;
  for (int c = tid; c < C; c += kThreads) s += expf(a[c] - amax);
  s = wave_sum(s);
  __syncthreads();
  if (l == 0) red[w] = s;
  __syncthreads();
  if (tid == 0) {
    float ss = 0.0f;
    for (int k = 0; k < kThreads / kWave; ++k) ss += red[k];
    bc[1] = ss;
  }
  __syncthreads();
  const float Z = bc[1];
  const int y = labels[b];
  const bool ok = y >= 0 && y < C;
  const float invB = 1.0f / (float)B;
  for (int c = tid; c < C; c += kThreads) {
    const float p = expf(a[c] - amax) / Z;
    dlda[(size_t)b * C + c] = (p - (c == y ? 1.0f : 0.0f)) * invB;
  }
  if (tid == 0) loss_b[b] = ok ? (logf(Z) - (a[y] - amax)) : NAN;
}

__global__ void ce_loss(const float* __restrict__ loss_b, int B, float* __restrict__ loss) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    float s = 0.0f;
    for (int b = 0; b < B; ++b) s += loss_b[b];
    *loss = s / (float)B;
  }
}

__global__ void fill_int(int32_t* __restrict__ p, size_t n, int32_t v) {
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) p[k] = v;
}

__global__ void ce_count(const int32_t* __restrict__ tstar, int B, int C, int32_t* __restrict__ counts) {
  const size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (k >= (size_t)B * C) return;
  const int b = (int)(k / C);
  atomicAdd(&counts[(size_t)tstar[k] * B + b], 1);
}

__global__ void ce_fill_max(const int32_t* __restrict__ tstar, const float* __restrict__ dlda, int B, int C,
                            const int32_t* __restrict__ row_ptr, int32_t* __restrict__ col_idx,
                            float* __restrict__ eps) {
  const size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (k >= (size_t)B * C) return;
  const int b = (int)(k / C);
  const int c = (int)(k - (size_t)b * C);
  const int t = tstar[k];
  int pos = 0;
  for (int c2 = 0; c2 < c; ++c2) pos += tstar[(size_t)b * C + c2] == t;
  const int64_t e = (int64_t)row_ptr[(size_t)t * B + b] + pos;
  col_idx[e] = c;
  eps[e] = dlda[k];
}

__global__ void ce_fill_sum(const float* __restrict__ dlda, int T, int B, int C, int32_t* __restrict__ row_ptr,
                            int32_t* __restrict__ col_idx, float* __restrict__ eps) {
  const size_t n = (size_t)T * B * C;
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    const size_t r = k / C;
    const int c = (int)(k - r * C);
    const int b = (int)(r % B);
    col_idx[k] = c;
    eps[k] = dlda[(size_t)b * C + c];
    if (c == 0) row_ptr[r] = (int32_t)k;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) row_ptr[(size_t)T * B] = (int32_t)n;
}

// dL/dV_out densely: dL/da at the arg-max time (mode 0) or at every t (mode 1), 0 elsewhere.
__global__ void ce_dense(const int32_t* __restrict__ tstar, const float* __restrict__ dlda, int T, int B, int C,
                         int mode, float* __restrict__ out) {
  const size_t n = (size_t)T * B * C;
  const size_t BC = (size_t)B * C;
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(k / BC);
    const size_t bc = k - (size_t)t * BC;
    out[k] = (mode == 1 || tstar[bc] == t) ? dlda[bc] : 0.0f;
  }
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" size_t snn_readout_ce_workspace(int T, int B, int C, int mode) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(C) || too_big(T, B, C) || (mode != 0 && mode != 1)) return 0;
  Carve c(nullptr);
  c.take<int32_t>((size_t)B * C);  // tstar
  c.take<float>((size_t)B * C);    // dL/da
  c.take<float>((size_t)B);        // per-sample loss
  c.take<int32_t>((size_t)T * B);  // row counts
  c.take<int32_t>(scan_temp_elems(T * B));
  c.take<int64_t>(1);
  return c.off;
}

extern "C" snn_status snn_readout_ce(const float* V_out, const int32_t* labels, int T, int B, int C, int mode,
                                     int32_t* row_ptr, int32_t* col_idx, float* eps, float* loss,
                                     float* eps_dense, void* workspace, size_t workspace_bytes, void* stream) {
  if (!V_out || !labels || !row_ptr || !col_idx || !eps || !loss || !workspace) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(C) || too_big(T, B, C)) return SNN_ERR_INVALID_ARG;
  if (mode != 0 && mode != 1) return SNN_ERR_INVALID_ARG;
  if (workspace_bytes < snn_readout_ce_workspace(T, B, C, mode)) return SNN_ERR_INVALID_ARG;
  if ((size_t)C * sizeof(float) > 64 * 1024) return SNN_ERR_UNSUPPORTED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carve ws(workspace);
  int32_t* tstar = ws.take<int32_t>((size_t)B * C);
  float* dlda = ws.take<float>((size_t)B * C);
  float* loss_b = ws.take<float>((size_t)B);
  int32_t* counts = ws.take<int32_t>((size_t)T * B);
  int32_t* temp = ws.take<int32_t>(scan_temp_elems(T * B));
  int64_t* nnz = ws.take<int64_t>(1);

  hipLaunchKernelGGL(ce_sample, dim3(B), dim3(kThreads), (size_t)C * sizeof(float), s, V_out, labels, T, B, C, mode,
                     tstar, dlda, loss_b);
  hipLaunchKernelGGL(ce_loss, dim3(1), dim3(64), 0, s, loss_b, B, loss);
  const size_t BC = (size_t)B * C;
  const unsigned gBC = (unsigned)((BC + 255) / 256);
  if (mode == 0) {
    const size_t rows = (size_t)T * B;
    hipLaunchKernelGGL(fill_int, dim3((unsigned)std::min<size_t>((rows + 255) / 256, 4096)), dim3(256), 0, s, counts,
                       rows, 0);
    hipLaunchKernelGGL(ce_count, dim3(gBC), dim3(256), 0, s, tstar, B, C, counts);
    launch_exclusive_scan(counts, T * B, row_ptr, nnz, temp, s);
    hipLaunchKernelGGL(ce_fill_max, dim3(gBC), dim3(256), 0, s, tstar, dlda, B, C, row_ptr, col_idx, eps);
  } else {
    const size_t n = (size_t)T * B * C;
    hipLaunchKernelGGL(ce_fill_sum, dim3((unsigned)std::min<size_t>((n + 255) / 256, 8192)), dim3(256), 0, s, dlda,
                       T, B, C, row_ptr, col_idx, eps);
  }
  if (eps_dense) {
    const size_t n = (size_t)T * B * C;
    hipLaunchKernelGGL(ce_dense, dim3((unsigned)std::min<size_t>((n + 255) / 256, 8192)), dim3(256), 0, s, tstar,
                       dlda, T, B, C, mode, eps_dense);
  }
  return launch_status();
}
