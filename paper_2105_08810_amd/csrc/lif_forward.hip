// LIF forward of one fully connected layer (Sec. 2.1): Eq. (lif) with V_rest = V_r = 0,
// V[0] = 0, the strict Heaviside of Eq. (spike_fn), and the input trace that Eq. (w_grad)
// reuses (the filtered input of Eq. (lif_unrolled)).
//
// Two kernels, so that no block walks the whole time axis with gathers on its critical path:
//   lif_gather  one wavefront per row (t, b), t < T-1: the ascending list of spiking inputs of
//               S_in[t,b,:] (ballots over 1024-input segments, list in LDS), then
//               I[t,b,:] = sum over that list of W[i,:], summed in ascending i. The row-parallel
//               sums have no dependence on time, so every row's W gathers can be in flight at
//               once. I[t,b,:] is parked in the slot of V[t+1,b,:].
//   lif_scan    one thread per (b, j): the membrane recurrence over t, reading I from V[t+1]
//               and overwriting it with V[t+1]; S_out[t] = V[t] > theta. And one thread per
//               (b, four inputs): the input trace over t. Loads run 16 steps ahead.
// Float32 with separately rounded operations (__fmul_rn / __fadd_rn) and the ascending
// summation order make V a deterministic function of the inputs.
#include "common.h"

namespace snn {
namespace {

constexpr int kGatherWaves = 4;        // wavefronts (rows) per gather block
constexpr int kPiece = 4 * kWave;      // inputs per ballot piece (4 bytes per lane)
constexpr int kSegPieces = 4;          // pieces whose spike bytes are loaded together
constexpr int kScanThreads = 256;
constexpr int kScanAhead = 32;         // time steps loaded ahead in the scans

template <bool ALIGNED>
__device__ __forceinline__ uint32_t load4(const uint8_t* p, int i, int n) {
  if (ALIGNED) return i < n ? *reinterpret_cast<const uint32_t*>(p + i) : 0u;
  uint32_t x = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (i + q < n) x |= (uint32_t)p[i + q] << (8 * q);
  return x;
}

// NQ float4 column groups per lane: lane l holds columns 4 (l + 64 m) .. +3, m < NQ.
// The row's spike bytes are read kSegPieces pieces at a time (all loads issued first), their
// spiking inputs listed in LDS in ascending order, and the list's W rows summed in batches.
template <bool ALIGNED, bool VEC, int NQ>
__global__ __launch_bounds__(kGatherWaves * kWave) void lif_gather(const uint8_t* __restrict__ s_in,
                                                                   const float* __restrict__ W, int T, int B,
                                                                   int N_in, int N_out, float* __restrict__ V) {
  constexpr int kBatch = NQ >= 16 ? 1 : (NQ >= 8 ? 2 : 4);  // W rows in flight: kBatch * NQ float4 loads
  __shared__ uint16_t seg_list[kGatherWaves][kSegPieces * kPiece];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const long r = (long)blockIdx.x * kGatherWaves + w;  // row r = t * B + b, t < T - 1
  if (r >= (long)(T - 1) * B) return;
  const uint8_t* row = s_in + (size_t)r * N_in;
  uint16_t* lst = seg_list[w];
  float acc[NQ][4];
#pragma unroll
  for (int m = 0; m < NQ; ++m)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[m][q] = 0.0f;

  for (int s0 = 0; s0 < N_in; s0 += kSegPieces * kPiece) {
    uint32_t x[kSegPieces];
#pragma unroll
    for (int c = 0; c < kSegPieces; ++c) x[c] = load4<ALIGNED>(row, s0 + c * kPiece + 4 * l, N_in);
    // ascending list of the segment's spiking inputs (offsets inside the segment)
    int base = 0;
#pragma unroll
    for (int c = 0; c < kSegPieces; ++c) {
      const bool a0 = (x[c] & 0xffu) != 0, a1 = (x[c] & 0xff00u) != 0, a2 = (x[c] & 0xff0000u) != 0,
                 a3 = (x[c] & 0xff000000u) != 0;
      const uint64_t m0 = __ballot(a0), m1 = __ballot(a1), m2 = __ballot(a2), m3 = __ballot(a3);
      int pos = base + mask_prefix(m0) + mask_prefix(m1) + mask_prefix(m2) + mask_prefix(m3);
      const int o = c * kPiece + 4 * l;
      if (a0) lst[pos++] = (uint16_t)o;
      if (a1) lst[pos++] = (uint16_t)(o + 1);
      if (a2) lst[pos++] = (uint16_t)(o + 2);
      if (a3) lst[pos++] = (uint16_t)(o + 3);
      base += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
    }
    const int n = base;
    __builtin_amdgcn_wave_barrier();
    // sums in ascending i, kBatch W rows in flight; positions past the list are clamped to its
    // last entry and their sums skipped by a select
    for (int k = 0; k < n; k += kBatch) {
      float4 wv[kBatch][NQ];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int ii = s0 + (int)lst[min(k + u, n - 1)];
        const float* wr = W + (size_t)ii * N_out;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          const int j = 4 * (l + kWave * m);
          if (VEC) {
            wv[u][m] = j < N_out ? *reinterpret_cast<const float4*>(wr + j) : make_float4(0.f, 0.f, 0.f, 0.f);
          } else {
            wv[u][m].x = j < N_out ? wr[j] : 0.0f;
            wv[u][m].y = j + 1 < N_out ? wr[j + 1] : 0.0f;
            wv[u][m].z = j + 2 < N_out ? wr[j + 2] : 0.0f;
            wv[u][m].w = j + 3 < N_out ? wr[j + 3] : 0.0f;
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const bool take = k + u < n;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          acc[m][0] = take ? __fadd_rn(acc[m][0], wv[u][m].x) : acc[m][0];
          acc[m][1] = take ? __fadd_rn(acc[m][1], wv[u][m].y) : acc[m][1];
          acc[m][2] = take ? __fadd_rn(acc[m][2], wv[u][m].z) : acc[m][2];
          acc[m][3] = take ? __fadd_rn(acc[m][3], wv[u][m].w) : acc[m][3];
        }
      }
    }
    __builtin_amdgcn_wave_barrier();  // the list is rewritten by the next segment
  }
  float* dst = V + (size_t)(r + B) * N_out;  // slot of V[t+1, b, :]
#pragma unroll
  for (int m = 0; m < NQ; ++m) {
    const int j = 4 * (l + kWave * m);
    if (VEC) {
      if (j < N_out) *reinterpret_cast<float4*>(dst + j) = make_float4(acc[m][0], acc[m][1], acc[m][2], acc[m][3]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (j + q < N_out) dst[j + q] = acc[m][q];
    }
  }
}

// Blocks [0, nv) run the membrane recurrence of B * N_out neurons; blocks [nv, nv + nt) run the
// trace of B * ceil(N_in / 4) input quads.
// With bits != NULL the recurrence also marks the active set of Definition 1: bit (t, k) of the
// bitset, k = b * N_out + j, is |V[t,b,j] - theta| < b_th in float32, word t * W64 + k / 64,
// W64 = ceil(B * N_out / 64); one ballot per wavefront and step (its 64 k are one word).
__device__ __forceinline__ void mark_active(uint64_t* bits, size_t word, bool valid, float v, float theta,
                                            float b_th) {
  const uint64_t m = __ballot(valid && fabsf(v - theta) < b_th);
  if (lane_id() == 0) bits[word] = m;
}

template <bool ALIGNED>
__global__ __launch_bounds__(kScanThreads) void lif_scan(const uint8_t* __restrict__ s_in, int T, int B, int N_in,
                                                         int N_out, float alpha, float theta, float b_th,
                                                         float* __restrict__ V, uint8_t* __restrict__ s_out,
                                                         float* __restrict__ trace, uint64_t* __restrict__ bits,
                                                         int nv) {
  if ((int)blockIdx.x < nv) {
    const size_t k0 = (size_t)blockIdx.x * kScanThreads + (threadIdx.x & ~(kWave - 1));
    if (k0 >= (size_t)B * N_out) return;  // whole wavefront past the end
    const size_t k = (size_t)blockIdx.x * kScanThreads + threadIdx.x;  // b * N_out + j
    const bool valid = k < (size_t)B * N_out;
    const size_t kc = valid ? k : k0;  // lanes past the end compute on a valid column, store nothing
    const size_t step = (size_t)B * N_out;
    const size_t W64 = (step + kWave - 1) / kWave;
    const size_t wword = k0 / kWave;
    float v = 0.0f;
    if (valid) V[k] = 0.0f;
    if (bits) mark_active(bits, wword, valid, v, theta, b_th);
    for (int t0 = 0; t0 < T - 1; t0 += kScanAhead) {
      const int np = min(kScanAhead, T - 1 - t0);
      float in[kScanAhead];
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) in[p] = V[(size_t)(t0 + min(p, np - 1) + 1) * step + kc];
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) {
        if (p < np) {
          const int t = t0 + p;
          const bool sp = v > theta;
          if (valid) s_out[(size_t)t * step + k] = (uint8_t)sp;
          v = __fadd_rn(__fadd_rn(__fmul_rn(alpha, v), in[p]), sp ? -1.0f : -0.0f);
          if (valid) V[(size_t)(t + 1) * step + k] = v;
          if (bits) mark_active(bits, (size_t)(t + 1) * W64 + wword, valid, v, theta, b_th);
        }
      }
    }
    if (valid) s_out[(size_t)(T - 1) * step + k] = (uint8_t)(v > theta);
  } else {
    const int nq = (N_in + 3) / 4;
    const size_t k = (size_t)(blockIdx.x - nv) * kScanThreads + threadIdx.x;  // b * nq + quad
    if (k >= (size_t)B * nq) return;
    const int b = (int)(k / nq);
    const int i = 4 * (int)(k - (size_t)b * nq);
    const size_t step = (size_t)B * N_in;
    float* dst0 = trace + (size_t)b * N_in + i;
    float tr[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (i + q < N_in) dst0[q] = 0.0f;
    const uint8_t* src0 = s_in + (size_t)b * N_in;
    for (int t0 = 0; t0 < T - 1; t0 += kScanAhead) {
      const int np = min(kScanAhead, T - 1 - t0);
      uint32_t x[kScanAhead];
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) x[p] = load4<ALIGNED>(src0 + (size_t)(t0 + min(p, np - 1)) * step, i, N_in);
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) {
        if (p < np) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            tr[q] = __fadd_rn(__fmul_rn(alpha, tr[q]), ((x[p] >> (8 * q)) & 0xffu) ? 1.0f : 0.0f);
          float* dst = dst0 + (size_t)(t0 + p + 1) * step;
          if (ALIGNED) {
            *reinterpret_cast<float4*>(dst) = make_float4(tr[0], tr[1], tr[2], tr[3]);
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
              if (i + q < N_in) dst[q] = tr[q];
          }
        }
      }
    }
  }
}

template <bool ALIGNED, bool VEC>
void launch_gather(int NQ, dim3 grid, hipStream_t s, const uint8_t* s_in, const float* W, int T, int B, int N_in,
                   int N_out, float* V) {
#define SNN_G(Q)                                                                                              \
  hipLaunchKernelGGL((lif_gather<ALIGNED, VEC, Q>), grid, dim3(kGatherWaves * kWave), 0, s, s_in, W, T, B, N_in, \
                     N_out, V)
  if (NQ <= 1) SNN_G(1);
  else if (NQ <= 2) SNN_G(2);
  else if (NQ <= 4) SNN_G(4);
  else if (NQ <= 8) SNN_G(8);
  else SNN_G(16);
#undef SNN_G
}

}  // namespace
}  // namespace snn

using namespace snn;

namespace {

// Convolutional LIF layer (3x3 filters, stride 1, zero padding 1, channels last): neuron
// k = b * N + n, n = (y * W + x) * F + f, N = H * W * F. Its weighted input at step t is the
// filter applied to the input spikes of the 3x3 patch, added in ascending input index
// (y', x', c) from +0.0 in separately rounded float32 adds (the order of the layer's Toeplitz
// matrix in the fully connected form), then the same recurrence and marking as lif_scan.
// WAVE_PIXEL (F a multiple of 64): a wavefront's 64 neurons share one pixel, so its lanes load
// the patch bytes of several steps at once (lane = (step, tap)), one ballot gives the spiking
// taps of those steps, and each lane adds its filter's weights for the set taps in tap order.
// Otherwise each lane forms its own patch sums, kConvAhead steps at a time.
constexpr int kConvAhead = 8;

template <bool WAVE_PIXEL>
__global__ __launch_bounds__(kScanThreads) void conv_scan(const uint8_t* __restrict__ s_in, const float* __restrict__ Wc,
                                                          int T, int B, int H, int W, int C, int F, float alpha,
                                                          float theta, float b_th, float* __restrict__ V,
                                                          uint8_t* __restrict__ s_out, uint64_t* __restrict__ bits) {
  const size_t N = (size_t)H * W * F;
  const size_t step = (size_t)B * N;
  const size_t k0 = (size_t)blockIdx.x * kScanThreads + (threadIdx.x & ~(kWave - 1));
  if (k0 >= step) return;  // whole wavefront past the end
  const size_t k = (size_t)blockIdx.x * kScanThreads + threadIdx.x;
  const bool valid = k < step;
  const size_t kc = valid ? k : k0;  // lanes past the end compute on a valid neuron, store nothing
  const int b = (int)(kc / N);
  const int n = (int)(kc - (size_t)b * N);
  const int f = n % F;
  const int pix = n / F;
  const int y = pix / W;
  const int x = pix - y * W;
  const size_t W64 = (step + kWave - 1) / kWave;
  const size_t wword = k0 / kWave;
  const size_t in_step = (size_t)B * H * W * C;
  const uint8_t* xb = s_in + (size_t)b * H * W * C;
  const int ntap = 9 * C;
  // WAVE_PIXEL: lane l < q * ntap loads tap (l % ntap) of step (l / ntap) of the group
  const int q = WAVE_PIXEL ? min(kConvAhead, kWave / ntap) : kConvAhead;
  const int l = lane_id();
  const int lp = l / ntap;
  const int ltap = l - lp * ntap;
  const int lky = ltap / (3 * C);
  const int lkx = (ltap / C) % 3;
  const int lc = ltap % C;
  const int lyy = y + lky - 1;
  const int lxx = x + lkx - 1;
  const bool lin = lp < q && lyy >= 0 && lyy < H && lxx >= 0 && lxx < W;
  const size_t loff = ((size_t)(lin ? lyy : 0) * W + (lin ? lxx : 0)) * C + lc;
  const uint64_t tapmask = ntap >= 64 ? ~0ull : ((1ull << ntap) - 1ull);
  float v = 0.0f;
  if (valid) V[k] = 0.0f;
  if (bits) mark_active(bits, wword, valid, v, theta, b_th);
  for (int t0 = 0; t0 < T - 1; t0 += q) {
    const int np = min(q, T - 1 - t0);
    float in[kConvAhead];
    if (WAVE_PIXEL) {
      const bool ld = lin && lp < np;
      const uint64_t m = __ballot(ld && xb[(size_t)(t0 + lp) * in_step + loff] != 0);
#pragma unroll
      for (int p = 0; p < kConvAhead; ++p) {
        float acc = 0.0f;
        if (p < np) {
          uint64_t taps = (m >> (p * ntap)) & tapmask;
          while (taps) {
            const int tap = __builtin_ctzll(taps);
            acc = __fadd_rn(acc, Wc[tap * F + f]);
            taps &= taps - 1ull;
          }
        }
        in[p] = acc;
      }
    } else {
#pragma unroll
      for (int p = 0; p < kConvAhead; ++p) {
        const uint8_t* xt = xb + (size_t)(t0 + min(p, np - 1)) * in_step;
        float acc = 0.0f;
        for (int ky = 0; ky < 3; ++ky) {
          const int yy = y + ky - 1;
          if (yy < 0 || yy >= H) continue;
          for (int kx = 0; kx < 3; ++kx) {
            const int xx = x + kx - 1;
            if (xx < 0 || xx >= W) continue;
            const uint8_t* px = xt + ((size_t)yy * W + xx) * C;
            for (int c = 0; c < C; ++c)
              if (px[c]) acc = __fadd_rn(acc, Wc[((ky * 3 + kx) * C + c) * F + f]);
          }
        }
        in[p] = acc;
      }
    }
#pragma unroll
    for (int p = 0; p < kConvAhead; ++p) {
      if (p < np) {
        const int t = t0 + p;
        const bool sp = v > theta;
        if (valid) s_out[(size_t)t * step + k] = (uint8_t)sp;
        v = __fadd_rn(__fadd_rn(__fmul_rn(alpha, v), in[p]), sp ? -1.0f : -0.0f);
        if (valid) V[(size_t)(t + 1) * step + k] = v;
        if (bits) mark_active(bits, (size_t)(t + 1) * W64 + wword, valid, v, theta, b_th);
      }
    }
  }
  if (valid) s_out[(size_t)(T - 1) * step + k] = (uint8_t)(v > theta);
}

snn_status lif_forward_impl(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out, float alpha,
                            float theta, float b_th, float* V, uint8_t* s_out, float* trace_in, uint64_t* bits,
                            void* stream) {
  if (!s_in || !W || !V || !s_out) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || isnan(theta)) return SNN_ERR_INVALID_ARG;
  if (bits && (isnan(b_th) || b_th < 0.0f)) return SNN_ERR_INVALID_ARG;
  if (N_out > 16 * 4 * kWave) return SNN_ERR_UNSUPPORTED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool al = (N_in % 4) == 0 && (reinterpret_cast<uintptr_t>(s_in) % 4) == 0;
  const bool vec = (N_out % 4) == 0 && (reinterpret_cast<uintptr_t>(W) % 16) == 0 &&
                   (reinterpret_cast<uintptr_t>(V) % 16) == 0;
  const int NQ = (N_out + 4 * kWave - 1) / (4 * kWave);
  const long rows = (long)(T - 1) * B;
  if (rows > 0) {
    const dim3 g((unsigned)((rows + kGatherWaves - 1) / kGatherWaves));
    if (al && vec) launch_gather<true, true>(NQ, g, s, s_in, W, T, B, N_in, N_out, V);
    else if (al) launch_gather<true, false>(NQ, g, s, s_in, W, T, B, N_in, N_out, V);
    else if (vec) launch_gather<false, true>(NQ, g, s, s_in, W, T, B, N_in, N_out, V);
    else launch_gather<false, false>(NQ, g, s, s_in, W, T, B, N_in, N_out, V);
  }
  const int nv = (int)(((size_t)B * N_out + kScanThreads - 1) / kScanThreads);
  const int nt = trace_in ? (int)(((size_t)B * ((N_in + 3) / 4) + kScanThreads - 1) / kScanThreads) : 0;
  const bool tal = al && (reinterpret_cast<uintptr_t>(trace_in) % 16) == 0;
  if (tal)
    hipLaunchKernelGGL(lif_scan<true>, dim3((unsigned)(nv + nt)), dim3(kScanThreads), 0, s, s_in, T, B, N_in, N_out,
                       alpha, theta, b_th, V, s_out, trace_in, bits, nv);
  else
    hipLaunchKernelGGL(lif_scan<false>, dim3((unsigned)(nv + nt)), dim3(kScanThreads), 0, s, s_in, T, B, N_in, N_out,
                       alpha, theta, b_th, V, s_out, trace_in, bits, nv);
  return launch_status();
}

}  // namespace

extern "C" snn_status snn_lif_forward(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                      float alpha, float theta, float* V, uint8_t* s_out, float* trace_in,
                                      void* stream) {
  return lif_forward_impl(s_in, W, T, B, N_in, N_out, alpha, theta, 0.0f, V, s_out, trace_in, nullptr, stream);
}

extern "C" size_t snn_active_bits_words(int T, int B, int N) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return 0;
  return (size_t)T * (((size_t)B * N + kWave - 1) / kWave);
}

extern "C" snn_status snn_lif_forward_active(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                             float alpha, float theta, float b_th, float* V, uint8_t* s_out,
                                             float* trace_in, uint64_t* active_bits, void* stream) {
  if (!active_bits) return SNN_ERR_INVALID_ARG;
  return lif_forward_impl(s_in, W, T, B, N_in, N_out, alpha, theta, b_th, V, s_out, trace_in, active_bits, stream);
}

extern "C" snn_status snn_conv_lif_forward(const uint8_t* s_in, const float* Wc, int T, int B, int H, int W, int C,
                                           int F, float alpha, float theta, float b_th, float* V, uint8_t* s_out,
                                           float* trace_in, uint64_t* active_bits, void* stream) {
  if (!s_in || !Wc || !V || !s_out) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(H) || bad_dim(W) || bad_dim(C) || bad_dim(F)) return SNN_ERR_INVALID_ARG;
  if ((int64_t)H * W * F >= ((int64_t)1 << 31) || (int64_t)H * W * C >= ((int64_t)1 << 31)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, H * W * F) || too_big(T, B, H * W * C)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || isnan(theta)) return SNN_ERR_INVALID_ARG;
  if (active_bits && (isnan(b_th) || b_th < 0.0f)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nv = (int)(((size_t)B * H * W * F + kScanThreads - 1) / kScanThreads);
  if (F % kWave == 0 && 9 * C <= kWave)  // a wavefront's lanes are the filters of one pixel
    hipLaunchKernelGGL(conv_scan<true>, dim3((unsigned)nv), dim3(kScanThreads), 0, s, s_in, Wc, T, B, H, W, C, F, alpha,
                       theta, b_th, V, s_out, active_bits);
  else
    hipLaunchKernelGGL(conv_scan<false>, dim3((unsigned)nv), dim3(kScanThreads), 0, s, s_in, Wc, T, B, H, W, C, F,
                       alpha, theta, b_th, V, s_out, active_bits);
  if (trace_in) {  // the input trace: lif_scan's trace blocks alone
    const int N_in = H * W * C;
    const int nt = (int)(((size_t)B * ((N_in + 3) / 4) + kScanThreads - 1) / kScanThreads);
    const bool tal = (N_in % 4) == 0 && (reinterpret_cast<uintptr_t>(s_in) % 4) == 0 &&
                     (reinterpret_cast<uintptr_t>(trace_in) % 16) == 0;
    if (tal)
      hipLaunchKernelGGL(lif_scan<true>, dim3((unsigned)nt), dim3(kScanThreads), 0, s, s_in, T, B, N_in, 1, alpha,
                         theta, b_th, nullptr, nullptr, trace_in, nullptr, 0);
    else
      hipLaunchKernelGGL(lif_scan<false>, dim3((unsigned)nt), dim3(kScanThreads), 0, s, s_in, T, B, N_in, 1, alpha,
                         theta, b_th, nullptr, nullptr, trace_in, nullptr, 0);
  }
  return launch_status();
}
