// Sparse backward of one LIF layer (Sec. 2.2): only active neurons carry gradient.
//
// dW (sparse form of Eq. (w_grad)): dW[:, j] += G[t,b,j] * trace[t,b,:] for every active
//   output entry (t,b,j), G = eps * g. A block owns a tile of TI input neurons for ALL output
//   neurons in LDS (layout [N_out][TI+1], so lanes over i hit distinct banks) and a chunk of
//   rows; each lane group streams the trace slice of one row and adds G*trace into column j
//   with LDS float64 atomics. Each block writes its tile once; a deterministic reduction over
//   row chunks produces dW. Trace bytes are read exactly once over the whole grid.
//
// grad_in (sparse form of Eq. (s_grad)): eps_in[t,b,i] = sum_j W[i,j] delta[t,b,j] at the
//   input layer's active entries, with delta[t] = alpha delta[t+1] + G[t+1] (Proposition 1's
//   memoised recurrence). Time is cut into C chunks so that B*C wavefronts walk in parallel:
//     chunk sums  L_c = sum_{t in c} alpha^(t - start_c) G[t]           (sparse, per (c,b))
//     carries     D_c = delta at the last step of chunk c, from D_{c+1} and L_{c+1}
//     walk        each (c,b) wavefront runs the recurrence from D_c down through its chunk,
//                 keeping delta[b, 0:N_out] in registers, and at every input-active entry
//                 gathers the W row and reduces W[i,:] . delta over the wavefront.
#include "common.h"

namespace snn {
namespace {

constexpr int kDwThreads = 1024;
constexpr int kRowsPerBatch = 32;
constexpr int kDwWaves = kDwThreads / kWave;
constexpr size_t kLdsBudget = 150 * 1024;
constexpr int kWalkThreads = 256;
constexpr int kWalkWaves = kWalkThreads / kWave;
constexpr int kGinBatch = 4;
constexpr int kAssumedCUs = 256;

struct DwPlan {
  int TI, n_itiles, n_chunks, rows_per_chunk;
  size_t lds;
};

DwPlan plan_dw(int T, int B, int N_in, int N_out) {
  DwPlan p{};
  const int TB = T * B;
  p.TI = 8;
  for (int ti : {64, 32, 16, 8}) {
    if ((size_t)N_out * (ti + 1) * sizeof(double) <= kLdsBudget) {
      p.TI = ti;
      break;
    }
  }
  p.lds = (size_t)N_out * (p.TI + 1) * sizeof(double);
  p.n_itiles = (N_in + p.TI - 1) / p.TI;
  const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(2, (160 * 1024) / p.lds));
  const int target = kAssumedCUs * per_cu;
  int nc = (target + p.n_itiles - 1) / p.n_itiles;
  nc = std::min(nc, std::max(1, TB / (4 * N_out)));  // partial tiles stay small next to the trace
  nc = std::min(nc, 64);
  nc = std::max(nc, 1);
  p.rows_per_chunk = (TB + nc - 1) / nc;
  p.n_chunks = (TB + p.rows_per_chunk - 1) / p.rows_per_chunk;
  return p;
}

struct WalkPlan {
  int P, C;
};

WalkPlan plan_walk(int T) {
  WalkPlan w{};
  w.P = std::max(4, std::min(64, (T + 15) / 16));
  w.C = (T + w.P - 1) / w.P;
  return w;
}

__device__ __forceinline__ int clamp_entry(int32_t v, int64_t cap) {
  return (int)(v < 0 ? 0 : (v > cap ? cap : v));
}

// ------------------------------------------------------------------ dW

__device__ __forceinline__ int rdlane(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
__device__ __forceinline__ float rdlane(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Each wavefront takes batches of kRowsPerBatch consecutive rows. G = 64/TI lane groups each
// own every G-th row of the batch; lane il of a group holds trace[r, i0 + il]. All loads of
// a batch (row pointers, trace slices, the first TI entries of every row) are issued before
// any is used, so a wavefront keeps a whole batch in flight; the entries are then broadcast
// inside each group with readlane (no LDS traffic besides the accumulation itself).
template <int TI, bool HAS_G>
__global__ __launch_bounds__(kDwThreads) void dw_tile_kernel(const float* __restrict__ trace, int TB, int N_in,
                                                             int N_out, const int32_t* __restrict__ row_ptr,
                                                             const int32_t* __restrict__ col_idx,
                                                             const float* __restrict__ g,
                                                             const float* __restrict__ eps, int64_t cap,
                                                             float* __restrict__ out, int rows_per_chunk,
                                                             int n_itiles) {
  // float64 accumulators: gfx950 executes ds_add_f64 about twenty times faster than ds_add_f32
  extern __shared__ double tile[];  // [N_out][TI + 1]
  constexpr int G = kWave / TI;
  constexpr int LD = TI + 1;
  constexpr int RB = (16 * G < kRowsPerBatch) ? 16 * G : kRowsPerBatch;  // rows per wavefront batch
  constexpr int KR = RB / G;                                            // rows per lane group
  const int it = blockIdx.x % n_itiles;
  const int c = blockIdx.x / n_itiles;
  const int i0 = it * TI;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int il = l % TI;
  const int sub = l / TI;
  const bool has_i = i0 + il < N_in;

  for (int k = tid; k < N_out * LD; k += kDwThreads) tile[k] = 0.0;
  __syncthreads();

  // Loads below are unconditional, from indices clamped into range, and masked afterwards with
  // selects: a branch around a load would make the compiler wait for it before the next one.
  const int r_lo = c * rows_per_chunk;
  const int r_hi = min(TB, r_lo + rows_per_chunk);
  const int ic = has_i ? i0 + il : 0;
  for (int rb = r_lo + w * RB; rb < r_hi; rb += kDwWaves * RB) {
    // row pointers first, then the trace slices: waiting for the former leaves the latter in flight
    const int rp_raw = row_ptr[min(rb + min(l, RB), r_hi)];
    float tr[KR];
#pragma unroll
    for (int k = 0; k < KR; ++k) tr[k] = trace[(size_t)min(rb + sub + G * k, r_hi - 1) * N_in + ic];
    __builtin_amdgcn_sched_barrier(0);
    const int rp = clamp_entry(rp_raw, cap);
#pragma unroll
    for (int k = 0; k < KR; ++k) tr[k] = (rb + sub + G * k < r_hi && has_i) ? tr[k] : 0.0f;
    int jv[KR];
    float ev[KR], gr[KR];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      const int q = sub + G * k;
      const int e0 = __shfl(rp, q, kWave);
      const int cnt = __shfl(rp, q + 1, kWave) - e0;
      const int e = il < cnt ? e0 + il : 0;  // cap >= 1 here; lanes past the row are masked later
      jv[k] = col_idx[e];
      ev[k] = eps[e];
      gr[k] = HAS_G ? g[e] : 1.0f;
    }
    __builtin_amdgcn_sched_barrier(0);  // keep every load of the batch ahead of any use
    float gv[KR];
#pragma unroll
    for (int k = 0; k < KR; ++k) gv[k] = ev[k] * gr[k];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      const int q = sub + G * k;
      const int e0 = __shfl(rp, q, kWave);
      const int cnt = __shfl(rp, q + 1, kWave) - e0;
      int mc = 0;
#pragma unroll
      for (int g2 = 0; g2 < G; ++g2) mc = max(mc, rdlane(cnt, g2 * TI));
      for (int base = 0; base < mc; base += TI) {
        if (base > 0) {  // rows longer than TI entries: next window
          const int e = base + il < cnt ? e0 + base + il : 0;
          const int jj = col_idx[e];
          const float ee = eps[e];
          const float gg = HAS_G ? g[e] : 1.0f;
          jv[k] = jj;
          gv[k] = ee * gg;
        }
        const int ns = min(TI, mc - base);
        for (int s = 0; s < ns; ++s) {
          int j = -1;
          float Gv = 0.0f;
#pragma unroll
          for (int g2 = 0; g2 < G; ++g2) {
            const int jj = rdlane(jv[k], g2 * TI + s);
            const float gg = rdlane(gv[k], g2 * TI + s);
            if (sub == g2) {
              j = jj;
              Gv = gg;
            }
          }
          if (base + s < cnt && (unsigned)j < (unsigned)N_out && has_i)
            atomicAdd(&tile[j * LD + il], (double)(Gv * tr[k]));
        }
      }
    }
  }
  __syncthreads();

  float* dst = out + (size_t)c * N_in * N_out;
  for (int k = tid; k < TI * N_out; k += kDwThreads) {
    const int ii = k / N_out;
    const int jj = k - ii * N_out;
    if (i0 + ii < N_in) dst[(size_t)(i0 + ii) * N_out + jj] = (float)tile[jj * LD + ii];
  }
}

__global__ void fill_zero(float* __restrict__ p, size_t n) {
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) p[k] = 0.0f;
}

__global__ void reduce_chunks(const float* __restrict__ part, int n_chunks, size_t n, float* __restrict__ out) {
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    float s = 0.0f;
    for (int c = 0; c < n_chunks; ++c) s += part[(size_t)c * n + k];
    out[k] = s;
  }
}

// ------------------------------------------------------------------ grad_in

// L[c][b][:] = sum_{t in chunk c} alpha^(t - start_c) G[t, b, :]   (sparse accumulation in LDS)
__global__ __launch_bounds__(kWalkThreads) void gin_chunk_sums(int T, int B, int N_out, float alpha, int P, int C,
                                                               const int32_t* __restrict__ row_ptr,
                                                               const int32_t* __restrict__ col_idx,
                                                               const float* __restrict__ g,
                                                               const float* __restrict__ eps, int64_t cap,
                                                               float* __restrict__ L) {
  extern __shared__ float sh[];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int q = blockIdx.x * kWalkWaves + w;
  if (q >= C * B) return;
  const int c = q / B;
  const int b = q - c * B;
  float* x = sh + (size_t)w * N_out;
  for (int j = l; j < N_out; j += kWave) x[j] = 0.0f;
  __builtin_amdgcn_wave_barrier();
  const int t_lo = c * P;
  const int t_hi = min(T, t_lo + P);
  float apow = 1.0f;
  for (int t = t_lo; t < t_hi; ++t) {
    const int r = t * B + b;
    const int e0 = clamp_entry(row_ptr[r], cap);
    const int e1 = clamp_entry(row_ptr[r + 1], cap);
    for (int e = e0 + l; e < e1; e += kWave) {  // distinct j inside a row: no two lanes collide
      const int j = col_idx[e];
      if ((unsigned)j < (unsigned)N_out) x[j] += apow * (eps[e] * (g ? g[e] : 1.0f));
    }
    __builtin_amdgcn_wave_barrier();
    apow *= alpha;
  }
  float* dst = L + (size_t)q * N_out;
  for (int j = l; j < N_out; j += kWave) dst[j] = x[j];
}

// In place over buf = L: buf[c] <- D_c (delta at the last step of chunk c), walking chunks
// from the last one, D_{C-1} = delta[T-1] = 0 and D_{c-1} = alpha^len_c D_c + L_c.
__global__ void gin_carries(int T, int B, int N_out, float alpha, int P, int C, float* __restrict__ buf) {
  const size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  const size_t BN = (size_t)B * N_out;
  if (k >= BN) return;
  float aP = 1.0f;
  for (int s = 0; s < P; ++s) aP *= alpha;
  const int last_len = T - (C - 1) * P;
  float aLast = 1.0f;
  for (int s = 0; s < last_len; ++s) aLast *= alpha;
  float x = 0.0f;
  for (int c = C - 1; c >= 0; --c) {
    const float Lc = buf[(size_t)c * BN + k];
    buf[(size_t)c * BN + k] = x;
    x = (c == C - 1 ? aLast : aP) * x + Lc;
  }
}

// One wavefront per (chunk c, sample b). delta[b, 0:N_out] lives in registers: lane l holds
// j = l + 64 m. The row pointers of all steps of the chunk are loaded once; at each step the
// input-active entries are taken kGinBatch at a time so that kGinBatch * NJ W loads are in
// flight, each reduced over the wavefront; then delta <- alpha delta + G[t] with the step's
// active outputs broadcast by readlane.
template <int NJ>
__global__ __launch_bounds__(kWalkThreads) void gin_walk(const float* __restrict__ W, int T, int B, int N_in,
                                                         int N_out, float alpha, int P, int C,
                                                         const int32_t* __restrict__ orp,
                                                         const int32_t* __restrict__ oci,
                                                         const float* __restrict__ og,
                                                         const float* __restrict__ oeps, int64_t ocap,
                                                         const int32_t* __restrict__ irp,
                                                         const int32_t* __restrict__ ici, int64_t icap,
                                                         const float* __restrict__ D, float* __restrict__ eps_in) {
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int q = blockIdx.x * kWalkWaves + w;
  if (q >= C * B) return;
  const int c = q / B;
  const int b = q - c * B;
  float d[NJ];
#pragma unroll
  for (int m = 0; m < NJ; ++m) {
    const int j = l + kWave * m;
    d[m] = j < N_out ? D[(size_t)q * N_out + j] : 0.0f;
  }
  const int t_lo = c * P;
  const int t_hi = min(T, t_lo + P);
  int ia = 0, ib = 0, oa = 0, ob = 0;
  if (l < t_hi - t_lo) {
    const int r = (t_lo + l) * B + b;
    ia = clamp_entry(irp[r], icap);
    ib = clamp_entry(irp[r + 1], icap);
    oa = clamp_entry(orp[r], ocap);
    ob = clamp_entry(orp[r + 1], ocap);
  }
  for (int t = t_hi - 1; t >= t_lo; --t) {
    const int k = t - t_lo;
    // eps_in at the input-active entries of row (t, b), with delta[t] = d
    const int i0 = rdlane(ia, k);
    const int i1 = rdlane(ib, k);
    for (int e = i0; e < i1; e += kGinBatch) {
      int iv[kGinBatch];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const int x = ici[min(e + u, i1 - 1)];
        iv[u] = (e + u < i1) ? x : -1;
      }
      float wv[kGinBatch][NJ];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const bool ok = (unsigned)iv[u] < (unsigned)N_in;
        const float* wr = W + (size_t)(ok ? iv[u] : 0) * N_out;
#pragma unroll
        for (int m = 0; m < NJ; ++m) {
          const int j = l + kWave * m;
          const float x = wr[min(j, N_out - 1)];
          wv[u][m] = (ok && j < N_out) ? x : 0.0f;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      float acc[kGinBatch];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        acc[u] = 0.0f;
#pragma unroll
        for (int m = 0; m < NJ; ++m) acc[u] += wv[u][m] * d[m];
      }
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const float s = wave_sum(acc[u]);
        if (l == 0 && e + u < i1) eps_in[e + u] = s;
      }
    }
    // delta[t-1] = alpha delta[t] + G[t]
#pragma unroll
    for (int m = 0; m < NJ; ++m) d[m] *= alpha;
    const int o0 = rdlane(oa, k);
    const int o1 = rdlane(ob, k);
    for (int e = o0; e < o1; e += kWave) {
      const int ec = min(e + l, o1 - 1);
      const int jj = oci[ec];
      const float ee = oeps[ec];
      const float gg = og ? og[ec] : 1.0f;
      const int jv = (e + l < o1) ? jj : -1;
      const float gv = ee * gg;
      const int ns = min(kWave, o1 - e);
      for (int s = 0; s < ns; ++s) {
        const int j = rdlane(jv, s);
        const float G = rdlane(gv, s);
        if ((unsigned)j < (unsigned)N_out) {
          const int jm = j / kWave;
          const bool mine = l == (j % kWave);
#pragma unroll
          for (int m = 0; m < NJ; ++m)
            if (m == jm && mine) d[m] += G;
        }
      }
    }
  }
}

template <int NJ>
void launch_walk(dim3 grid, size_t lds, hipStream_t s, const float* W, int T, int B, int N_in, int N_out,
                 float alpha, int P, int C, const int32_t* orp, const int32_t* oci, const float* og,
                 const float* oeps, int64_t ocap, const int32_t* irp, const int32_t* ici, int64_t icap,
                 const float* D, float* eps_in) {
  hipLaunchKernelGGL(gin_walk<NJ>, grid, dim3(kWalkThreads), lds, s, W, T, B, N_in, N_out, alpha, P, C, orp, oci,
                     og, oeps, ocap, irp, ici, icap, D, eps_in);
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" size_t snn_sparse_backward_workspace(int T, int B, int N_in, int N_out) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return 0;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return 0;
  const DwPlan p = plan_dw(T, B, N_in, N_out);
  const WalkPlan wp = plan_walk(T);
  Carve c(nullptr);
  if (p.n_chunks > 1) c.take<float>((size_t)p.n_chunks * N_in * N_out);
  c.take<float>((size_t)wp.C * B * N_out);
  return c.off;
}

extern "C" snn_status snn_sparse_backward(const float* W, const float* trace_in, int T, int B, int N_in, int N_out,
                                          float alpha, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                                          const float* out_g, const float* eps_out, int64_t out_cap,
                                          const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap,
                                          float* eps_in, float* dW, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  if (!W || !trace_in || !out_row_ptr || !dW) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || out_cap < 0 || in_cap < 0) return SNN_ERR_INVALID_ARG;
  if (out_cap > 0 && (!out_col_idx || !eps_out)) return SNN_ERR_INVALID_ARG;
  const bool grad_in = in_row_ptr != nullptr;
  if (grad_in && in_cap > 0 && (!in_col_idx || !eps_in)) return SNN_ERR_INVALID_ARG;
  if (!grad_in && (in_col_idx || eps_in)) return SNN_ERR_INVALID_ARG;
  const size_t need = snn_sparse_backward_workspace(T, B, N_in, N_out);
  if (need > 0 && (!workspace || workspace_bytes < need)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  const int TB = T * B;
  const DwPlan p = plan_dw(T, B, N_in, N_out);
  const WalkPlan wp = plan_walk(T);
  Carve ws(workspace);
  float* part = p.n_chunks > 1 ? ws.take<float>((size_t)p.n_chunks * N_in * N_out) : dW;
  float* Lbuf = ws.take<float>((size_t)wp.C * B * N_out);

  const dim3 dgrid((unsigned)(p.n_itiles * p.n_chunks));
  if (out_cap == 0) {  // no active entry: dW = 0, and no entry array may be read
    hipLaunchKernelGGL(fill_zero, dim3((unsigned)std::min<size_t>(((size_t)N_in * N_out + 255) / 256, 4096)),
                       dim3(256), 0, s, dW, (size_t)N_in * N_out);
    return launch_status();
  }
#define SNN_DW2(TI_, HG_)                                                                                 \
  do {                                                                                                     \
    (void)hipFuncSetAttribute((const void*)dw_tile_kernel<TI_, HG_>,                                       \
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);                     \
    hipLaunchKernelGGL((dw_tile_kernel<TI_, HG_>), dgrid, dim3(kDwThreads), p.lds, s, trace_in, TB, N_in,  \
                       N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, part, p.rows_per_chunk,   \
                       p.n_itiles);                                                                        \
  } while (0)
#define SNN_DW(TI_)             \
  do {                          \
    if (out_g)                  \
      SNN_DW2(TI_, true);       \
    else                        \
      SNN_DW2(TI_, false);      \
  } while (0)
  switch (p.TI) {
    case 64: SNN_DW(64); break;
    case 32: SNN_DW(32); break;
    case 16: SNN_DW(16); break;
    default: SNN_DW(8); break;
  }
#undef SNN_DW
  if (p.n_chunks > 1) {
    const size_t n = (size_t)N_in * N_out;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(reduce_chunks, dim3(blocks), dim3(256), 0, s, part, p.n_chunks, n, dW);
  }

  if (grad_in && in_cap > 0) {
    const int pairs = wp.C * B;
    const dim3 wgrid((pairs + kWalkWaves - 1) / kWalkWaves);
    const size_t lds = (size_t)kWalkWaves * N_out * sizeof(float);  // chunk sums only
    hipLaunchKernelGGL(gin_chunk_sums, wgrid, dim3(kWalkThreads), lds, s, T, B, N_out, alpha, wp.P, wp.C,
                       out_row_ptr, out_col_idx, out_g, eps_out, out_cap, Lbuf);
    const size_t BN = (size_t)B * N_out;
    hipLaunchKernelGGL(gin_carries, dim3((unsigned)((BN + 255) / 256)), dim3(256), 0, s, T, B, N_out, alpha, wp.P,
                       wp.C, Lbuf);
    const int nj = (N_out + kWave - 1) / kWave;
#define SNN_WALK(NJ_)                                                                                         \
  launch_walk<NJ_>(wgrid, 0, s, W, T, B, N_in, N_out, alpha, wp.P, wp.C, out_row_ptr, out_col_idx, out_g, \
                   eps_out, out_cap, in_row_ptr, in_col_idx, in_cap, Lbuf, eps_in)
    if (nj <= 1) SNN_WALK(1);
    else if (nj <= 2) SNN_WALK(2);
    else if (nj <= 4) SNN_WALK(4);
    else if (nj <= 8) SNN_WALK(8);
    else if (nj <= 16) SNN_WALK(16);
    else if (nj <= 32) SNN_WALK(32);
    else SNN_WALK(64);
#undef SNN_WALK
  }
  return launch_status();
}
