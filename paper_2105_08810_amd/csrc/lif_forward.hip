// LIF forward of one fully connected layer (Sec. 2.1): Eq. (lif) with V_rest = V_r = 0,
// V[0] = 0, the strict Heaviside of Eq. (spike_fn), and the input trace that Eq. (w_grad)
// reuses (the filtered input of Eq. (lif_unrolled)).
//
// The weighted input of a row (t, b) is I[t,b,:] = sum of W[i,:] over the row's spiking inputs,
// added in ascending i (the list of spiking inputs comes from ballots over the row's bytes), and
// the recurrence V[t+1] = (alpha V[t] + I[t]) - S_out[t], S_out[t] = V[t] > theta, walks time per
// neuron. Two forms:
//   lif_fused   (the default) one block per (sample, group of columns) walks time in tiles: its
//               wavefronts form a tile's weighted inputs two rows each into LDS, then every
//               thread runs its column's recurrence over the tile from LDS. V, S_out, the active
//               bitset and the input trace are written once; the weighted inputs never reach HBM.
//               The trace of the output spikes (the next layer's input trace) can be written
//               beside V from the spike bits the recurrence has in hand.
//   lif_gather + lif_scan  (widths whose bitset words straddle samples, W rows that are not
//               whole float4 columns, grids of fewer than two blocks per CU) one wavefront per row
//               parks I[t,b,:] in the slot of V[t+1,b,:]; then one thread per (b, j) runs the
//               recurrence over t, overwriting it with V[t+1], and one thread per (b, input) the
//               input trace.
// Float32 with separately rounded operations (__fmul_rn / __fadd_rn) and the ascending
// summation order make V a deterministic function of the inputs; both forms give the same bits.
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

// The spike bytes of one segment of a row (kSegPieces pieces of 4 bytes per lane; bytes past
// N_in read as no spike).
template <bool ALIGNED>
__device__ __forceinline__ void load_segment(const uint8_t* __restrict__ row, int s0, int N_in,
                                             uint32_t (&x)[kSegPieces]) {
  const int l = lane_id();
#pragma unroll
  for (int c = 0; c < kSegPieces; ++c) x[c] = load4<ALIGNED>(row, s0 + c * kPiece + 4 * l, N_in);
}

// Ascending list (offsets inside the segment) of a segment's spiking inputs in lst; returns its
// length.
__device__ __forceinline__ int segment_list(const uint32_t (&x)[kSegPieces], uint16_t* lst) {
  const int l = lane_id();
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
  return base;
}

// Ascending list of a segment's spiking inputs as byte offsets inside their piece (piece c's
// entries at [starts[c], starts[c + 1]) of lst); returns its length.
__device__ __forceinline__ int segment_list8(const uint32_t (&x)[kSegPieces], uint8_t* lst, int (&starts)[kSegPieces]) {
  const int l = lane_id();
  int base = 0;
#pragma unroll
  for (int c = 0; c < kSegPieces; ++c) {
    starts[c] = base;
    const bool a0 = (x[c] & 0xffu) != 0, a1 = (x[c] & 0xff00u) != 0, a2 = (x[c] & 0xff0000u) != 0,
               a3 = (x[c] & 0xff000000u) != 0;
    const uint64_t m0 = __ballot(a0), m1 = __ballot(a1), m2 = __ballot(a2), m3 = __ballot(a3);
    int pos = base + mask_prefix(m0) + mask_prefix(m1) + mask_prefix(m2) + mask_prefix(m3);
    const int o = 4 * l;
    if (a0) lst[pos++] = (uint8_t)o;
    if (a1) lst[pos++] = (uint8_t)(o + 1);
    if (a2) lst[pos++] = (uint8_t)(o + 2);
    if (a3) lst[pos++] = (uint8_t)(o + 3);
    base += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
  }
  return base;
}

// Input index of list entry e (s0: the segment's first input).
__device__ __forceinline__ int list8_input(const uint8_t* lst, const int (&starts)[kSegPieces], int e, int s0) {
  const int c = (e >= starts[1]) + (e >= starts[2]) + (e >= starts[3]);
  return s0 + c * kPiece + (int)lst[e];
}

// The weighted input of one row (t, b) at NQ float4 column groups per lane: lane l sums columns
// col0 + 4 (l + 64 m) .. +3, m < NQ, over the row's spiking inputs in ascending i, from +0.0 with
// separately rounded adds. The row's spike bytes are read kSegPieces pieces at a time (all loads
// issued first), their spiking inputs listed in lst (LDS) in ascending order, and the list's W
// rows summed KB at a time (KB * NQ float4 loads in flight).
template <bool ALIGNED, bool VEC, int NQ, int KB>
__device__ __forceinline__ void row_input_sums(const uint8_t* __restrict__ row, const float* __restrict__ W, int N_in,
                                               int N_out, int col0, uint16_t* lst, float (&acc)[NQ][4]) {
  const int l = lane_id();
#pragma unroll
  for (int m = 0; m < NQ; ++m)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[m][q] = 0.0f;

  for (int s0 = 0; s0 < N_in; s0 += kSegPieces * kPiece) {
    uint32_t x[kSegPieces];
    load_segment<ALIGNED>(row, s0, N_in, x);
    const int n = segment_list(x, lst);
    __builtin_amdgcn_wave_barrier();
    // sums in ascending i, KB W rows in flight; positions past the list are clamped to its last
    // entry and their sums skipped by a select
    for (int k = 0; k < n; k += KB) {
      float4 wv[KB][NQ];
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const int ii = s0 + (int)lst[min(k + u, n - 1)];
        const float* wr = W + (size_t)ii * N_out + col0;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          const int j = 4 * (l + kWave * m);
          const int jn = N_out - col0;  // columns of the row from col0 on
          if (VEC) {
            wv[u][m] = j < jn ? *reinterpret_cast<const float4*>(wr + j) : make_float4(0.f, 0.f, 0.f, 0.f);
          } else {
            wv[u][m].x = j < jn ? wr[j] : 0.0f;
            wv[u][m].y = j + 1 < jn ? wr[j + 1] : 0.0f;
            wv[u][m].z = j + 2 < jn ? wr[j + 2] : 0.0f;
            wv[u][m].w = j + 3 < jn ? wr[j + 3] : 0.0f;
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < KB; ++u) {
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
}

// One wavefront per row (t, b), t < T - 1: the row's weighted input over every column, parked in
// the slot of V[t+1, b, :].
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
  float acc[NQ][4];
  row_input_sums<ALIGNED, VEC, NQ, kBatch>(s_in + (size_t)r * N_in, W, N_in, N_out, 0, seg_list[w], acc);
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

// The input trace of input k = b * N_in + i over the whole time axis: trace[0] = 0,
// trace[t+1] = alpha trace[t] + S_in[t] (loads kScanAhead steps ahead). One input per lane, not
// four: four times the wavefronts for the same bytes, so that more of them overlap their load and
// store phases (T = 500, B = 256, 1024 inputs: 0.152 -> 0.123 ms beside the recurrence).
__device__ __forceinline__ void trace_walk(size_t k, const uint8_t* __restrict__ s_in, int T, int B, int N_in,
                                           float alpha, float* __restrict__ trace) {
  const size_t step = (size_t)B * N_in;
  if (k >= step) return;
  float tr = 0.0f;
  trace[k] = 0.0f;
  for (int t0 = 0; t0 < T - 1; t0 += kScanAhead) {
    const int np = min(kScanAhead, T - 1 - t0);
    uint32_t x[kScanAhead];
#pragma unroll
    for (int p = 0; p < kScanAhead; ++p) x[p] = s_in[(size_t)(t0 + min(p, np - 1)) * step + k];
#pragma unroll
    for (int p = 0; p < kScanAhead; ++p) {
      if (p < np) {
        tr = __fadd_rn(__fmul_rn(alpha, tr), x[p] ? 1.0f : 0.0f);
        trace[(size_t)(t0 + p + 1) * step + k] = tr;
      }
    }
  }
}

// The input trace of input quad k = b * ceil(N_in / 4) + quad over the whole time axis, as
// trace_walk (the trace blocks beside lif_fused's blocks: there four inputs per lane are faster,
// 0.326 against 0.340 ms at T = 100, B = 512, 2312 inputs).
template <bool ALIGNED>
__device__ __forceinline__ void trace_walk4(size_t k, const uint8_t* __restrict__ s_in, int T, int B, int N_in,
                                            float alpha, float* __restrict__ trace) {
  const int nq = (N_in + 3) / 4;
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

// Blocks [0, nv) run the membrane recurrence of B * N_out neurons; blocks [nv, nv + nt) run the
// trace of B * N_in inputs.
// With bits != NULL the recurrence also marks the active set of Definition 1: bit (t, k) of the
// bitset, k = b * N_out + j, is |V[t,b,j] - theta| < b_th in float32, word t * W64 + k / 64,
// W64 = ceil(B * N_out / 64); one ballot per wavefront and step (its 64 k are one word).
__device__ __forceinline__ void mark_active(uint64_t* bits, size_t word, bool valid, float v, float theta,
                                            float b_th) {
  const uint64_t m = __ballot(valid && fabsf(v - theta) < b_th);
  if (lane_id() == 0) bits[word] = m;
}

__global__ __launch_bounds__(kScanThreads) void lif_scan(const uint8_t* __restrict__ s_in, int T, int B, int N_in,
                                                         int N_out, float alpha, float theta, float b_th,
                                                         float* __restrict__ V, uint8_t* __restrict__ s_out,
                                                         float* __restrict__ trace, float* __restrict__ trace_out,
                                                         float alpha_next, uint64_t* __restrict__ bits, int nv) {
  if ((int)blockIdx.x < nv) {
    const size_t k0 = (size_t)blockIdx.x * kScanThreads + (threadIdx.x & ~(kWave - 1));
    if (k0 >= (size_t)B * N_out) return;  // whole wavefront past the end
    const size_t k = (size_t)blockIdx.x * kScanThreads + threadIdx.x;  // b * N_out + j
    const bool valid = k < (size_t)B * N_out;
    const size_t kc = valid ? k : k0;  // lanes past the end compute on a valid column, store nothing
    const size_t step = (size_t)B * N_out;
    const size_t W64 = (step + kWave - 1) / kWave;
    const size_t wword = k0 / kWave;
    float v = 0.0f, to = 0.0f;
    if (valid) V[k] = 0.0f;
    if (trace_out && valid) trace_out[k] = 0.0f;
    if (bits) mark_active(bits, wword, valid, v, theta, b_th);
    // Two groups of kScanAhead steps in flight: a group's loads are issued before the previous
    // group's stores, so waiting for them (the memory counter retires in order) does not wait
    // for those stores as well. A group's loads read slots no earlier store writes.
    auto load = [&](float (&in)[kScanAhead], int t0) {
      const int np = min(kScanAhead, T - 1 - t0);
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) in[p] = V[(size_t)(t0 + min(p, np - 1) + 1) * step + kc];
    };
    auto walk = [&](const float (&in)[kScanAhead], int t0) {
      const int np = min(kScanAhead, T - 1 - t0);
#pragma unroll
      for (int p = 0; p < kScanAhead; ++p) {
        if (p < np) {
          const int t = t0 + p;
          const bool sp = v > theta;
          if (valid) s_out[(size_t)t * step + k] = (uint8_t)sp;
          v = __fadd_rn(__fadd_rn(__fmul_rn(alpha, v), in[p]), sp ? -1.0f : -0.0f);
          if (valid) V[(size_t)(t + 1) * step + k] = v;
          if (trace_out) {
            to = __fadd_rn(__fmul_rn(alpha_next, to), sp ? 1.0f : 0.0f);
            if (valid) trace_out[(size_t)(t + 1) * step + k] = to;
          }
          if (bits) mark_active(bits, (size_t)(t + 1) * W64 + wword, valid, v, theta, b_th);
        }
      }
    };
    float ina[kScanAhead], inb[kScanAhead];
    if (T > 1) load(ina, 0);
    for (int t0 = 0; t0 < T - 1; t0 += 2 * kScanAhead) {
      const int t1 = t0 + kScanAhead;
      if (t1 < T - 1) load(inb, t1);
      walk(ina, t0);
      if (t1 < T - 1) {
        if (t1 + kScanAhead < T - 1) load(ina, t1 + kScanAhead);
        walk(inb, t1);
      }
    }
    if (valid) s_out[(size_t)(T - 1) * step + k] = (uint8_t)(v > theta);
  } else {
    trace_walk((size_t)(blockIdx.x - nv) * kScanThreads + threadIdx.x, s_in, T, B, N_in, alpha, trace);
  }
}

// The weighted inputs of two rows at once (the sums and order of row_input_sums for each): the
// rows' spike lists are formed segment by segment and their W rows summed together, KB of each
// row in flight. x0 / x1 hold the first segment's spike bytes (loaded by the caller ahead of
// time); a null row has no spikes.
template <bool ALIGNED, int NQ, int KB>
__device__ __forceinline__ void row_pair_sums(const uint8_t* r0, const uint8_t* r1, const uint32_t (&x0)[kSegPieces],
                                              const uint32_t (&x1)[kSegPieces], const float* __restrict__ W,
                                              int N_in, int N_out, int col0, uint8_t* lst0, uint8_t* lst1,
                                              float (&acc0)[NQ][4], float (&acc1)[NQ][4]) {
  const int l = lane_id();
  const int jn = N_out - col0;  // columns of a W row from col0 on (a multiple of 4)
#pragma unroll
  for (int m = 0; m < NQ; ++m)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc0[m][q] = acc1[m][q] = 0.0f;
  for (int s0 = 0; s0 < N_in; s0 += kSegPieces * kPiece) {
    uint32_t y0[kSegPieces], y1[kSegPieces];
#pragma unroll
    for (int c = 0; c < kSegPieces; ++c) y0[c] = y1[c] = 0u;
    if (s0 == 0) {
#pragma unroll
      for (int c = 0; c < kSegPieces; ++c) {
        y0[c] = x0[c];
        y1[c] = x1[c];
      }
    } else {
      if (r0) load_segment<ALIGNED>(r0, s0, N_in, y0);
      if (r1) load_segment<ALIGNED>(r1, s0, N_in, y1);
    }
    int st0[kSegPieces], st1[kSegPieces];
    const int n0 = segment_list8(y0, lst0, st0);
    const int n1 = segment_list8(y1, lst1, st1);
    __builtin_amdgcn_wave_barrier();
    const int n = max(n0, n1);
    for (int k = 0; k < n; k += KB) {
      float4 wa[KB][NQ], wb[KB][NQ];
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const int i0 = n0 > 0 ? list8_input(lst0, st0, min(k + u, n0 - 1), s0) : s0;
        const int i1 = n1 > 0 ? list8_input(lst1, st1, min(k + u, n1 - 1), s0) : s0;
        const float* w0 = W + (size_t)i0 * N_out + col0;
        const float* w1 = W + (size_t)i1 * N_out + col0;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          const int j = 4 * (l + kWave * m);
          wa[u][m] = j < jn ? *reinterpret_cast<const float4*>(w0 + j) : make_float4(0.f, 0.f, 0.f, 0.f);
          wb[u][m] = j < jn ? *reinterpret_cast<const float4*>(w1 + j) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const bool t0 = k + u < n0, t1 = k + u < n1;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          acc0[m][0] = t0 ? __fadd_rn(acc0[m][0], wa[u][m].x) : acc0[m][0];
          acc0[m][1] = t0 ? __fadd_rn(acc0[m][1], wa[u][m].y) : acc0[m][1];
          acc0[m][2] = t0 ? __fadd_rn(acc0[m][2], wa[u][m].z) : acc0[m][2];
          acc0[m][3] = t0 ? __fadd_rn(acc0[m][3], wa[u][m].w) : acc0[m][3];
          acc1[m][0] = t1 ? __fadd_rn(acc1[m][0], wb[u][m].x) : acc1[m][0];
          acc1[m][1] = t1 ? __fadd_rn(acc1[m][1], wb[u][m].y) : acc1[m][1];
          acc1[m][2] = t1 ? __fadd_rn(acc1[m][2], wb[u][m].z) : acc1[m][2];
          acc1[m][3] = t1 ? __fadd_rn(acc1[m][3], wb[u][m].w) : acc1[m][3];
        }
      }
    }
    __builtin_amdgcn_wave_barrier();  // the lists are rewritten by the next segment
  }
}

// Fused forward. Blocks [0, nfb): one per (sample b, column group cg of JW = 256 NQ columns),
// walking the time axis in tiles of kFuseP = 2 kFuseWaves steps. In a tile each wavefront forms the
// weighted inputs of two of the tile's rows (row_pair_sums) in an LDS tile; after a barrier each
// thread runs the membrane recurrence of its column over the tile's steps from the LDS tile, so
// V, S_out and the active bitset are written once and the weighted inputs never reach HBM; the
// spike bytes of the next tile's rows are requested before the recurrence. Blocks [nfb, ...):
// the input trace, one thread per input quad (trace_walk4), beside them. Bit-identical to
// lif_gather + lif_scan. With a bitset each wavefront's 64 columns must be one bitset word
// (N_out % 64 == 0, checked by the caller).
constexpr int kFuseThreads = 512;
constexpr int kFuseWaves = kFuseThreads / kWave;
constexpr int kFuseP = 2 * kFuseWaves;  // steps per tile: two rows per wavefront

template <bool ALIGNED, int NQ, bool STASH, bool TOUT>
__global__ __launch_bounds__(kFuseThreads) __attribute__((amdgpu_waves_per_eu(4))) void lif_fused(
    const uint8_t* __restrict__ s_in, const float* __restrict__ W, int T, int B, int N_in, int N_out, int G, int nfb,
    float alpha, float theta, float b_th, float* __restrict__ V, uint8_t* __restrict__ s_out,
    float* __restrict__ trace, float* __restrict__ trace_out, float alpha_next, uint64_t* __restrict__ bits) {
  constexpr int JW = 4 * kWave * NQ;  // columns of a group
  constexpr int KB = NQ >= 2 ? 4 : 8;
  static_assert(JW <= kFuseThreads, "one scan thread per column of the group");
  static_assert(!STASH || ALIGNED, "stashed spike bytes are whole input quads");
  if (!STASH && (int)blockIdx.x >= nfb) {
    trace_walk4<ALIGNED>((size_t)(blockIdx.x - nfb) * kFuseThreads + threadIdx.x, s_in, T, B, N_in, alpha, trace);
    return;
  }
  __shared__ __attribute__((aligned(16))) float tile[kFuseP][JW];
  __shared__ uint8_t lists[2 * kFuseWaves][kSegPieces * kPiece];
  // STASH (N_in <= one segment): the tile's spike bytes, input quad q of step p at [p][q], for the trace
  __shared__ uint32_t rowbytes[STASH ? kFuseP : 1][kSegPieces * kWave];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int b = blockIdx.x / G;
  const int cg = blockIdx.x - b * G;
  const int c0 = cg * JW;
  const size_t vstep = (size_t)B * N_out;
  const size_t W64 = (vstep + kWave - 1) / kWave;
  const size_t istep = (size_t)B * N_in;
  // scan thread k: column c0 + k of sample b; wavefronts whose first column is past N_out skip
  const int k = threadIdx.x;
  const int kw = k - l;  // the wavefront's first column slot
  const bool scan_wave = kw < JW && c0 + kw < N_out;
  const bool valid = scan_wave && c0 + k < N_out;
  const size_t vk = (size_t)b * N_out + c0 + (valid ? k : kw);
  const size_t wword = ((size_t)b * N_out + c0 + kw) / kWave;
  // rows w and w + kFuseWaves of tile t0 (null past T - 2)
  auto row_of = [&](int t0, int p) -> const uint8_t* {
    const int t = t0 + p;
    return t < T - 1 ? s_in + (size_t)t * istep + (size_t)b * N_in : nullptr;
  };
  uint32_t x0[kSegPieces], x1[kSegPieces];
  auto prefetch = [&](int t0) {
    const uint8_t* r0 = row_of(t0, w);
    const uint8_t* r1 = row_of(t0, w + kFuseWaves);
#pragma unroll
    for (int c = 0; c < kSegPieces; ++c) x0[c] = x1[c] = 0u;
    if (r0) load_segment<ALIGNED>(r0, 0, N_in, x0);
    if (r1) load_segment<ALIGNED>(r1, 0, N_in, x1);
  };
  // STASH: the trace of the group's input quads, thread k taking quad q_lo + k
  const int nq = (N_in + 3) / 4;
  const int qpg = (nq + G - 1) / G;
  const int tq = (cg * qpg + k < nq && k < qpg) ? cg * qpg + k : -1;
  float tr[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (STASH && trace && tq >= 0)
    *reinterpret_cast<float4*>(trace + (size_t)b * N_in + 4 * tq) = make_float4(0.f, 0.f, 0.f, 0.f);
  float v = 0.0f, to = 0.0f;
  if (valid) V[vk] = 0.0f;
  if (TOUT && valid) trace_out[vk] = 0.0f;
  if (bits && scan_wave) mark_active(bits, wword, valid, v, theta, b_th);
  prefetch(0);
  for (int t0 = 0; t0 < T - 1; t0 += kFuseP) {
    const int np = min(kFuseP, T - 1 - t0);
    if (STASH) {
#pragma unroll
      for (int c = 0; c < kSegPieces; ++c) {
        rowbytes[w][c * kWave + l] = x0[c];
        rowbytes[w + kFuseWaves][c * kWave + l] = x1[c];
      }
    }
    {
      float acc0[NQ][4], acc1[NQ][4];
      row_pair_sums<ALIGNED, NQ, KB>(row_of(t0, w), row_of(t0, w + kFuseWaves), x0, x1, W, N_in, N_out, c0,
                                     lists[w], lists[w + kFuseWaves], acc0, acc1);
#pragma unroll
      for (int m = 0; m < NQ; ++m) {
        const int j = 4 * (l + kWave * m);
        *reinterpret_cast<float4*>(&tile[w][j]) = make_float4(acc0[m][0], acc0[m][1], acc0[m][2], acc0[m][3]);
        *reinterpret_cast<float4*>(&tile[w + kFuseWaves][j]) =
            make_float4(acc1[m][0], acc1[m][1], acc1[m][2], acc1[m][3]);
      }
    }
    __syncthreads();
    prefetch(t0 + kFuseP);  // in flight during the recurrence
    if (scan_wave) {
#pragma unroll
      for (int p = 0; p < kFuseP; ++p) {
        if (p < np) {
          const int t = t0 + p;
          const bool sp = v > theta;
          if (valid) s_out[(size_t)t * vstep + vk] = (uint8_t)sp;
          v = __fadd_rn(__fadd_rn(__fmul_rn(alpha, v), tile[p][k]), sp ? -1.0f : -0.0f);
          if (valid) V[(size_t)(t + 1) * vstep + vk] = v;
          if (TOUT) {
            to = __fadd_rn(__fmul_rn(alpha_next, to), sp ? 1.0f : 0.0f);
            if (valid) trace_out[(size_t)(t + 1) * vstep + vk] = to;
          }
          if (bits) mark_active(bits, (size_t)(t + 1) * W64 + wword, valid, v, theta, b_th);
        }
      }
    }
    if (STASH && trace && tq >= 0) {
      float* dst0 = trace + (size_t)b * N_in + 4 * tq;
#pragma unroll
      for (int p = 0; p < kFuseP; ++p) {
        if (p < np) {
          const uint32_t x = rowbytes[p][tq];
#pragma unroll
          for (int q = 0; q < 4; ++q) tr[q] = __fadd_rn(__fmul_rn(alpha, tr[q]), ((x >> (8 * q)) & 0xffu) ? 1.0f : 0.0f);
          *reinterpret_cast<float4*>(dst0 + (size_t)(t0 + p + 1) * istep) = make_float4(tr[0], tr[1], tr[2], tr[3]);
        }
      }
    }
    __syncthreads();  // the tile is rewritten by the next tile's sums
  }
  if (valid) s_out[(size_t)(T - 1) * vstep + vk] = (uint8_t)(v > theta);
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
                            float theta, float b_th, float* V, uint8_t* s_out, float* trace_in, float* trace_out,
                            float alpha_next, uint64_t* bits, void* stream) {
  if (!s_in || !W || !V || !s_out) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out)) return SNN_ERR_INVALID_ARG;
  if (too_big(T, B, N_in) || too_big(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || isnan(theta)) return SNN_ERR_INVALID_ARG;
  if (bits && (isnan(b_th) || b_th < 0.0f)) return SNN_ERR_INVALID_ARG;
  if (trace_out && bad_alpha(alpha_next)) return SNN_ERR_INVALID_ARG;
  if (N_out > 16 * 4 * kWave) return SNN_ERR_UNSUPPORTED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool al = (N_in % 4) == 0 && (reinterpret_cast<uintptr_t>(s_in) % 4) == 0;
  {  // the fused kernel: whole float4 W columns, whole bitset words per wavefront, a 16-byte aligned trace,
     // and at least two blocks per CU (with fewer, its time walk is latency-bound and the two-kernel
     // form is faster: a 1024 -> 100 readout at T = 500, B = 256, 5% input spikes, takes 0.61 against
     // 0.46 ms)
    const int fq = N_out > 4 * kWave ? 2 : 1;
    const int G = (N_out + 4 * kWave * fq - 1) / (4 * kWave * fq);
    if ((N_out % 4) == 0 && (reinterpret_cast<uintptr_t>(W) % 16) == 0 && (!bits || N_out % kWave == 0) &&
        (!trace_in || !al || (reinterpret_cast<uintptr_t>(trace_in) % 16) == 0) &&
        (int64_t)B * G >= 2 * (int64_t)cu_count()) {
      // the trace from the tile's stashed spike bytes when a row is one segment and the group's input
      // quads fit one per thread; otherwise trace blocks beside the fused blocks
      const bool stash = al && N_in <= kSegPieces * kPiece && ((N_in + 3) / 4 + G - 1) / G <= kFuseThreads;
      const int nfb = B * G;
      const int ntb = (trace_in && !stash) ? (int)(((size_t)B * ((N_in + 3) / 4) + kFuseThreads - 1) / kFuseThreads) : 0;
      const dim3 g((unsigned)(nfb + ntb));
#define SNN_F(A, Q, ST)                                                                                              \
  do {                                                                                                               \
    if (trace_out)                                                                                                   \
      hipLaunchKernelGGL((lif_fused<A, Q, ST, true>), g, dim3(kFuseThreads), 0, s, s_in, W, T, B, N_in, N_out, G,     \
                         nfb, alpha, theta, b_th, V, s_out, trace_in, trace_out, alpha_next, bits);                  \
    else                                                                                                             \
      hipLaunchKernelGGL((lif_fused<A, Q, ST, false>), g, dim3(kFuseThreads), 0, s, s_in, W, T, B, N_in, N_out, G,    \
                         nfb, alpha, theta, b_th, V, s_out, trace_in, nullptr, 1.0f, bits);                          \
  } while (0)
      if (stash && fq == 2) SNN_F(true, 2, true);
      else if (stash) SNN_F(true, 1, true);
      else if (al && fq == 2) SNN_F(true, 2, false);
      else if (al) SNN_F(true, 1, false);
      else if (fq == 2) SNN_F(false, 2, false);
      else SNN_F(false, 1, false);
#undef SNN_F
      return launch_status();
    }
  }
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
  const int nt = trace_in ? (int)(((size_t)B * N_in + kScanThreads - 1) / kScanThreads) : 0;
  hipLaunchKernelGGL(lif_scan, dim3((unsigned)(nv + nt)), dim3(kScanThreads), 0, s, s_in, T, B, N_in, N_out, alpha,
                     theta, b_th, V, s_out, trace_in, trace_out, alpha_next, bits, nv);
  return launch_status();
}

}  // namespace

extern "C" snn_status snn_lif_forward(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                      float alpha, float theta, float* V, uint8_t* s_out, float* trace_in,
                                      void* stream) {
  return lif_forward_impl(s_in, W, T, B, N_in, N_out, alpha, theta, 0.0f, V, s_out, trace_in, nullptr, 1.0f,
                          nullptr, stream);
}

extern "C" size_t snn_active_bits_words(int T, int B, int N) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return 0;
  return (size_t)T * (((size_t)B * N + kWave - 1) / kWave);
}

extern "C" snn_status snn_lif_forward_active(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                             float alpha, float theta, float b_th, float* V, uint8_t* s_out,
                                             float* trace_in, uint64_t* active_bits, void* stream) {
  if (!active_bits) return SNN_ERR_INVALID_ARG;
  return lif_forward_impl(s_in, W, T, B, N_in, N_out, alpha, theta, b_th, V, s_out, trace_in, nullptr, 1.0f,
                          active_bits, stream);
}

extern "C" snn_status snn_lif_forward_traces(const uint8_t* s_in, const float* W, int T, int B, int N_in,
                                             int N_out, float alpha, float theta, float b_th, float* V,
                                             uint8_t* s_out, float* trace_in, float* trace_out,
                                             float alpha_next, uint64_t* active_bits, void* stream) {
  return lif_forward_impl(s_in, W, T, B, N_in, N_out, alpha, theta, b_th, V, s_out, trace_in, trace_out, alpha_next,
                          active_bits, stream);
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
    const int nt = (int)(((size_t)B * N_in + kScanThreads - 1) / kScanThreads);
    hipLaunchKernelGGL(lif_scan, dim3((unsigned)nt), dim3(kScanThreads), 0, s, s_in, T, B, N_in, 1, alpha, theta,
                       b_th, nullptr, nullptr, trace_in, nullptr, 1.0f, nullptr, 0);
  }
  return launch_status();
}
