// Sparse backward of one LIF layer (Sec. 2.2): only active neurons carry gradient.
//
// dW (sparse form of Eq. (w_grad)): dW[:, j] += G[t,b,j] * trace[t,b,:] for every active
//   output entry (t,b,j), G = eps * g. A block owns 128 input neurons (two per lane) times a
//   slab of up to kSlab output neurons in LDS as float64 accumulators ([slab][129]), and a
//   chunk of rows. A wavefront streams the 256-byte trace slices of a batch of rows, finds
//   each row's entries inside the slab with two ballots (column indices are ascending inside
//   a row), and adds G*trace into the slab row by row; every entry is uniform across the
//   wavefront, so one float64 LDS atomic covers 64 multiply-adds. Blocks write their slab
//   once; a fixed-order reduction over row chunks produces dW.
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
constexpr int kRowsPerBatch = 8;  // rows a wavefront has in flight
constexpr int kSlab = 128;        // output neurons per LDS slab
constexpr int kNi = 2;            // input neurons per lane: lane l holds inputs l and l + 64 of its tile
constexpr int kItile = kNi * kWave;
constexpr int kLd = kItile + 1;   // padded slab row: 128 inputs + 1
constexpr int kDwWaves = kDwThreads / kWave;
constexpr size_t kLdsBudget = 150 * 1024;
constexpr int kWalkThreads = 256;
constexpr int kWalkWaves = kWalkThreads / kWave;
constexpr int kGinBatch = 4;
constexpr int kAssumedCUs = 256;
constexpr int kBufWord3 = 0x00020000;  // buffer descriptor word 3 on gfx9: 32-bit data format

struct DwPlan {
  int n_itiles, n_slabs, slab, n_chunks, rows_per_chunk;
  size_t lds;
};

DwPlan plan_dw(int T, int B, int N_in, int N_out) {
  DwPlan p{};
  const int TB = T * B;
  p.n_slabs = (N_out + kSlab - 1) / kSlab;
  p.slab = (N_out + p.n_slabs - 1) / p.n_slabs;
  p.lds = (size_t)p.slab * kLd * sizeof(double);
  p.n_itiles = (N_in + kItile - 1) / kItile;
  const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(2, (160 * 1024) / p.lds));
  const int target = kAssumedCUs * per_cu * 8;  // short chunks: the slab blocks of a tile stay close (L2 reuse)
  const int tiles = p.n_itiles * p.n_slabs;
  int nc = (target + tiles - 1) / tiles;
  nc = std::min(nc, std::max(1, TB / (4 * N_out)));  // partial slabs stay small next to the trace
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
  w.P = std::max(4, std::min(64, (T + 31) / 32));
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

// Slab-major copy of the active entries. For slab s and row r, sp[s*TB + r] is where row r's
// entries with s*slab <= j < (s+1)*slab start; each record holds the entry's byte offset inside
// its slab row of the LDS accumulator and G = eps * g.
struct SlabRec {
  int32_t off;
  float G;
};

// A wavefront takes R consecutive rows (R * n_slabs <= 64): their entries are contiguous in the
// CSR, and lane k of each 64-entry piece finds its entry's row from the batch's row pointers.
// An entry's key is (row in batch, slab); with ascending columns the entries of one key are a
// run of lanes, and a run's head is found with one ballot. Per-key totals live in a 64-int LDS
// array of the wavefront (runs may continue into the next piece). Entries whose column is
// outside [0, N_out) are neither counted nor placed.
constexpr int kRowWaves = 4;

struct EntryKey {
  int key;    // row-in-batch * n_slabs + slab, or -1
  int j;      // column
  int h;      // lane of the run's first entry in this piece
  bool tail;  // last lane of the run in this piece
};

__device__ __forceinline__ EntryKey entry_key(int ee, int E1, int rp, int nr, int N_out, int n_slabs, int slab,
                                              const int32_t* __restrict__ col_idx) {
  const int l = lane_id();
  EntryKey x{-1, -1, 0, false};
  if (ee < E1) {
    x.j = col_idx[ee];
    if ((unsigned)x.j < (unsigned)N_out) {
      int k = 0;
      for (int m = 1; m < nr; ++m) k += ee >= rdlane(rp, m);
      x.key = k * n_slabs + x.j / slab;
    }
  }
  const int prev = __shfl_up(x.key, 1, kWave);
  const int next = __shfl_down(x.key, 1, kWave);
  const bool head = x.key >= 0 && (l == 0 || prev != x.key);
  x.tail = x.key >= 0 && (l == kWave - 1 || next != x.key);
  const uint64_t le = __ballot(head) & ((2ull << l) - 1ull);  // heads at or below this lane
  x.h = le ? 63 - __clzll(le) : 0;
  return x;
}

__global__ __launch_bounds__(kRowWaves * kWave) void slab_count(int TB, int N_out, int n_slabs, int slab, int R,
                                                                const int32_t* __restrict__ row_ptr,
                                                                const int32_t* __restrict__ col_idx, int64_t cap,
                                                                int32_t* __restrict__ cnt) {
  __shared__ int tot[kRowWaves][kWave];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int r0 = (blockIdx.x * kRowWaves + w) * R;
  if (r0 >= TB) return;
  const int nr = min(R, TB - r0);
  int* tw = tot[w];
  tw[l] = 0;
  const int rp = l <= nr ? clamp_entry(row_ptr[r0 + l], cap) : 0;
  const int E0 = rdlane(rp, 0);
  const int E1 = rdlane(rp, nr);
  for (int e = E0; e < E1; e += kWave) {
    const EntryKey x = entry_key(e + l, E1, rp, nr, N_out, n_slabs, slab, col_idx);
    if (x.tail) tw[x.key] += l - x.h + 1;
  }
  if (l < nr * n_slabs) cnt[(size_t)(l % n_slabs) * TB + r0 + l / n_slabs] = tw[l];
}

template <bool HAS_G>
__global__ __launch_bounds__(kRowWaves * kWave) void slab_fill(int TB, int N_out, int n_slabs, int slab, int R,
                                                               const int32_t* __restrict__ row_ptr,
                                                               const int32_t* __restrict__ col_idx,
                                                               const float* __restrict__ g,
                                                               const float* __restrict__ eps, int64_t cap,
                                                               const int32_t* __restrict__ sp, int64_t nrec,
                                                               SlabRec* __restrict__ rec) {
  __shared__ int done[kRowWaves][kWave];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int r0 = (blockIdx.x * kRowWaves + w) * R;
  if (r0 >= TB) return;
  const int nr = min(R, TB - r0);
  int* dw = done[w];
  dw[l] = 0;
  const int rp = l <= nr ? clamp_entry(row_ptr[r0 + l], cap) : 0;
  const int E0 = rdlane(rp, 0);
  const int E1 = rdlane(rp, nr);
  // lane p: first slot of key p (row r0 + p / n_slabs in slab p % n_slabs)
  const int first = l < nr * n_slabs ? sp[(size_t)(l % n_slabs) * TB + r0 + l / n_slabs] : 0;
  for (int e = E0; e < E1; e += kWave) {
    const int ee = e + l;
    const EntryKey x = entry_key(ee, E1, rp, nr, N_out, n_slabs, slab, col_idx);
    const int kq = x.key >= 0 ? x.key : 0;
    const int pos = __shfl(first, kq, kWave) + dw[kq] + (l - x.h);
    if (x.key >= 0 && pos < nrec) {
      const int sl = kq % n_slabs;
      SlabRec r;
      r.off = (x.j - sl * slab) * kLd * (int)sizeof(double);
      r.G = eps[ee] * (HAS_G ? g[ee] : 1.0f);
      rec[pos] = r;
    }
    if (x.tail) dw[x.key] += l - x.h + 1;
  }
}

// Block (c, it, sl): inputs [128 it, 128 it + 128), outputs of slab sl, rows of chunk c. Lane l
// holds inputs 128 it + l and 128 it + 64 + l, so one record read, conversion and address serve
// two float64 LDS atomics (the second at an immediate offset): on this hardware the VALU work of
// an atomic adds to its LDS time instead of overlapping it. Blocks of one chunk are numbered so
// that they land on one XCD and share its L2 lines.
__global__ __launch_bounds__(kDwThreads) void dw_slab_kernel(const float* __restrict__ trace, int TB, int N_in,
                                                             int N_out, const int32_t* __restrict__ sp,
                                                             const SlabRec* __restrict__ rec, int64_t nrec,
                                                             float* __restrict__ out, int rows_per_chunk,
                                                             int n_itiles, int n_slabs, int slab) {
  extern __shared__ double acc[];  // [slab][kLd]
  int id = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) id = (id & 7) * (nb >> 3) + (id >> 3);
  const int tiles = n_itiles * n_slabs;
  const int c = id / tiles;
  const int sl = (id - c * tiles) % n_slabs;  // the slabs of one input tile run side by side and
  const int it = (id - c * tiles) / n_slabs;  // read the same trace slices (L2 hits)
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int i0 = it * kItile + l;
  const int ic0 = min(i0, N_in - 1);  // lanes past N_in accumulate rows that are never written out
  const int ic1 = min(i0 + kWave, N_in - 1);
  const int j0 = sl * slab;
  const int j1 = min(N_out, j0 + slab);
  const int32_t* spl = sp + (size_t)sl * TB;
  char* accb = reinterpret_cast<char*>(acc) + l * (int)sizeof(double);
  const int max_off = (slab - 1) * kLd * (int)sizeof(double);

  for (int k = tid; k < slab * kLd; k += kDwThreads) acc[k] = 0.0;
  __syncthreads();

  const int r_lo = c * rows_per_chunk;
  const int r_hi = min(TB, r_lo + rows_per_chunk);
  const int2* rec2 = reinterpret_cast<const int2*>(rec);
  // Software pipeline over batches of 8 rows: while a batch is processed, the next batch's
  // trace values and records are in flight and the row pointers of the one after it. Rows past
  // r_hi read sp[r_hi] (empty ranges); a row with no entry in this slab reads the chunk's first
  // trace row instead of its own (a cache hit, never used).
  auto load_sp = [&](int rb) { return spl[min(rb + min(l, kRowsPerBatch), r_hi)]; };
  auto load_rest = [&](int rb, int spv, float* t0, float* t1, int2& ra) {
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      const bool any = rdlane(spv, k + 1) > rdlane(spv, k);
      const size_t row = (size_t)(any ? min(rb + k, r_hi - 1) : r_lo) * N_in;
      t0[k] = trace[row + ic0];
      t1[k] = trace[row + ic1];
    }
    ra = rec2[min((int64_t)rdlane(spv, 0) + l, nrec - 1)];  // lane s holds the batch's record s
  };
  constexpr int kStride = kDwWaves * kRowsPerBatch;
  int rb = r_lo + w * kRowsPerBatch;
  int spv = load_sp(rb);
  float tr0[kRowsPerBatch], tr1[kRowsPerBatch];
  int2 ra;
  load_rest(rb, spv, tr0, tr1, ra);
  int spv_n = load_sp(rb + kStride);
  for (; rb < r_hi; rb += kStride) {
    float tn0[kRowsPerBatch], tn1[kRowsPerBatch];
    int2 ran;
    load_rest(rb + kStride, spv_n, tn0, tn1, ran);
    const int spv_nn = load_sp(rb + 2 * kStride);
    __builtin_amdgcn_sched_barrier(0);
    const int base = rdlane(spv, 0);
    const int n = rdlane(spv, kRowsPerBatch) - base;
    if (n <= kWave) {  // common case: the batch's records are all in one register
      int lo = 0;
#pragma unroll
      for (int k = 0; k < kRowsPerBatch; ++k) {
        const double t0 = (double)tr0[k], t1 = (double)tr1[k];
        const int hi = rdlane(spv, k + 1) - base;
        for (int s = lo; s < hi; ++s) {
          const int off = (int)min((unsigned)rdlane(ra.x, s), (unsigned)max_off);  // scalar clamp into the slab
          const double G = (double)__int_as_float(rdlane(ra.y, s));
          double* a = reinterpret_cast<double*>(accb + off);
          atomicAdd(a, t0 * G);
          atomicAdd(a + kWave, t1 * G);
        }
        lo = hi;
      }
    } else {  // dense batch: records read one by one (uniform addresses)
#pragma unroll
      for (int k = 0; k < kRowsPerBatch; ++k) {
        const double t0 = (double)tr0[k], t1 = (double)tr1[k];
        const int lo = rdlane(spv, k);
        const int hi = rdlane(spv, k + 1);
        for (int s = lo; s < hi; ++s) {
          const int2 x = rec2[min((int64_t)s, nrec - 1)];  // clamped: malformed input cannot read past the records
          const double G = (double)__int_as_float(x.y);
          double* a = reinterpret_cast<double*>(accb + min(max(x.x, 0), max_off));
          atomicAdd(a, t0 * G);
          atomicAdd(a + kWave, t1 * G);
        }
      }
    }
    spv = spv_n;
    spv_n = spv_nn;
    ra = ran;
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      tr0[k] = tn0[k];
      tr1[k] = tn1[k];
    }
  }
  __syncthreads();
  float* dst = out + (size_t)c * N_in * N_out;
  const int width = j1 - j0;
  for (int k = tid; k < kItile * width; k += kDwThreads) {
    const int ii = k / width;
    const int jj = k - ii * width;
    if (it * kItile + ii < N_in) dst[(size_t)(it * kItile + ii) * N_out + j0 + jj] = (float)acc[jj * kLd + ii];
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

// Buffer descriptor of one row of n floats (raw buffer, range-checked: reads past the row give 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const float* row, int n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), (short)0, n * (int)sizeof(float), kBufWord3);
}

// One float through a buffer descriptor (the builtin returns the raw 32 bits).
__device__ __forceinline__ float load_f32(__amdgpu_buffer_rsrc_t rs, int byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, byte_off, 0, 0));
}

// Sum over the wavefront of four values at once (one per entry u): two exchanges across
// halves and across rows leave each 16-lane row holding entry u = row index summed over 4
// lanes; four DPP steps then finish the sum inside the row. Returns the total of entry
// (lane >> 4) in every lane of that row.
__device__ __forceinline__ float wave_sum4(float a0, float a1, float a2, float a3) {
  const int l = lane_id();
  const bool b5 = (l >> 5) & 1;
  const bool b4 = (l >> 4) & 1;
  const float s0 = b5 ? a0 : a2, s1 = b5 ? a1 : a3;
  const float k0 = b5 ? a2 : a0, k1 = b5 ? a3 : a1;
  const float c0 = k0 + __shfl_xor(s0, 32, kWave);
  const float c1 = k1 + __shfl_xor(s1, 32, kWave);
  float v = (b4 ? c1 : c0) + __shfl_xor(b4 ? c0 : c1, 16, kWave);
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, true));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, true));  // row_mirror
  return v;
}

// One wavefront per (chunk c, sample b). delta[b, 0:N_out] lives in registers: lane l holds
// j = l + 64 m. The row pointers of all steps of the chunk are loaded once, and each step's
// entry indices (input and output side, one entry per lane) are requested one step ahead, so
// that a step waits only for its W rows. The input-active entries are taken four at a time
// (4 * NJ W loads in flight) and reduced together; then delta <- alpha delta + G[t], each
// active output added by the lane that owns its column (a uniform register index).
template <int NJ>
__global__ __launch_bounds__(kWalkThreads, NJ <= 16 ? 4 : 1) void gin_walk(const float* __restrict__ W, int T, int B, int N_in,
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
  // grid-stride over (c, b): a grid smaller than C*B/4 blocks leaves room on every CU for
  // other work (the dW kernel on another stream)
  for (int q = blockIdx.x * kWalkWaves + w; q < C * B; q += gridDim.x * kWalkWaves) {
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
  // entry l of step k's row (clamped into the row; only lanes below the row length are used)
  auto in_idx = [&](int k) {
    const int a = rdlane(ia, k), z = rdlane(ib, k);
    return z > a ? ici[min(a + l, z - 1)] : -1;
  };
  auto out_col = [&](int k) {
    const int a = rdlane(oa, k), z = rdlane(ob, k);
    return z > a ? oci[min(a + l, z - 1)] : -1;
  };
  auto out_g = [&](int k) {
    const int a = rdlane(oa, k), z = rdlane(ob, k);
    const int e = min(a + l, max(z - 1, 0));
    return z > a ? oeps[e] * (og ? og[e] : 1.0f) : 0.0f;
  };
  int k = t_hi - 1 - t_lo;
  int vi = in_idx(k), vj = out_col(k);
  float vg = out_g(k);
  for (; k >= 0; --k) {
    const int kn = max(k - 1, 0);
    const int vi_n = in_idx(kn), vj_n = out_col(kn);
    const float vg_n = out_g(kn);
    // eps_in at the input-active entries of row (t, b), with delta[t] = d
    const int i0 = rdlane(ia, k);
    const int i1 = rdlane(ib, k);
    for (int e = i0; e < i1; e += kGinBatch) {
      int iv[kGinBatch];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const int eu = e + u;
        const int x = eu - i0 < kWave ? rdlane(vi, min(eu - i0, kWave - 1)) : ici[min(eu, i1 - 1)];
        iv[u] = (eu < i1 && (unsigned)x < (unsigned)N_in) ? x : -1;
      }
      // W row gathers through a buffer descriptor per row (base in scalar registers, column
      // offsets as immediates, columns past N_out read as 0 by the range check)
      float wv[kGinBatch][NJ];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const __amdgpu_buffer_rsrc_t rs = row_rsrc(W + (size_t)(iv[u] >= 0 ? iv[u] : 0) * N_out, N_out);
#pragma unroll
        for (int m = 0; m < NJ; ++m) wv[u][m] = load_f32(rs, (l + kWave * m) * 4);
      }
      __builtin_amdgcn_sched_barrier(0);
      float acc[kGinBatch];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        acc[u] = 0.0f;
#pragma unroll
        for (int m = 0; m < NJ; ++m) acc[u] += wv[u][m] * d[m];  // d = 0 past N_out
        acc[u] = iv[u] >= 0 ? acc[u] : 0.0f;
      }
      const float tot = wave_sum4(acc[0], acc[1], acc[2], acc[3]);
      const int u = l >> 4;
      if ((l & 15) == 0 && e + u < i1) eps_in[e + u] = tot;
    }
    // delta[t-1] = alpha delta[t] + G[t]
#pragma unroll
    for (int m = 0; m < NJ; ++m) d[m] *= alpha;
    const int o0 = rdlane(oa, k);
    const int o1 = rdlane(ob, k);
    for (int e = o0; e < o1; e += kWave) {
      int jv = vj;
      float gv = vg;
      if (e > o0) {  // rows with more than 64 active outputs: the rest is read here
        const int ec = min(e + l, o1 - 1);
        jv = oci[ec];
        gv = oeps[ec] * (og ? og[ec] : 1.0f);
      }
      const int ns = min(kWave, o1 - e);
      for (int s = 0; s < ns; ++s) {
        const int j = rdlane(jv, s);
        const float G = rdlane(gv, s);
        if ((unsigned)j < (unsigned)N_out) {
          const int jm = j / kWave;  // uniform: a register index, not a branch per m
          d[jm] += (l == j % kWave) ? G : 0.0f;
        }
      }
    }
    vi = vi_n;
    vj = vj_n;
    vg = vg_n;
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

namespace snn {
namespace {

size_t dw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap) {
  const DwPlan p = plan_dw(T, B, N_in, N_out);
  const int nsp = p.n_slabs * T * B;
  Carve c(nullptr);
  if (p.n_chunks > 1) c.take<float>((size_t)p.n_chunks * N_in * N_out);
  c.take<int32_t>((size_t)nsp + 1);
  c.take<int32_t>((size_t)nsp);
  c.take<int32_t>(scan_temp_elems(nsp));
  c.take<SlabRec>((size_t)std::max<int64_t>(out_cap, 1));
  return c.off;
}

size_t gin_workspace(int T, int B, int N_out) {
  const WalkPlan wp = plan_walk(T);
  Carve c(nullptr);
  c.take<float>((size_t)wp.C * B * N_out);
  return c.off;
}

bool dims_ok(int T, int B, int N_in, int N_out) {
  return !(bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(N_out) || too_big(T, B, N_in) ||
           too_big(T, B, N_out));
}

void fill_zero_async(float* p, size_t n, hipStream_t s) {
  if (n == 0) return;
  hipLaunchKernelGGL(fill_zero, dim3((unsigned)std::min<size_t>((n + 255) / 256, 4096)), dim3(256), 0, s, p, n);
}

// dW of one layer: group-major records of the active entries, the slab accumulation, the
// reduction over row chunks. Arguments already validated.
void enqueue_dw(const float* trace_in, int T, int B, int N_in, int N_out, const int32_t* out_row_ptr,
                const int32_t* out_col_idx, const float* out_g, const float* eps_out, int64_t out_cap, float* dW,
                void* workspace, hipStream_t s) {
  if (out_cap == 0) {  // no active output entry: dW = 0 and no entry array is read
    fill_zero_async(dW, (size_t)N_in * N_out, s);
    return;
  }
  const int TB = T * B;
  const DwPlan p = plan_dw(T, B, N_in, N_out);
  Carve ws(workspace);
  float* part = p.n_chunks > 1 ? ws.take<float>((size_t)p.n_chunks * N_in * N_out) : dW;
  const int nsp = p.n_slabs * TB;
  int32_t* sp = ws.take<int32_t>((size_t)nsp + 1);
  int32_t* scnt = ws.take<int32_t>((size_t)nsp);
  int32_t* stmp = ws.take<int32_t>(scan_temp_elems(nsp));
  SlabRec* rec = ws.take<SlabRec>((size_t)std::max<int64_t>(out_cap, 1));

  const int R = std::max(1, std::min(8, kWave / p.n_slabs));  // rows per wavefront
  const int nwaves = (TB + R - 1) / R;
  const dim3 rgrid((unsigned)((nwaves + kRowWaves - 1) / kRowWaves));
  const dim3 rblock(kRowWaves * kWave);
  const int64_t nrec = std::max<int64_t>(out_cap, 1);
  hipLaunchKernelGGL(slab_count, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr, out_col_idx,
                     out_cap, scnt);
  launch_exclusive_scan(scnt, nsp, sp, nullptr, stmp, s);
  if (out_g)
    hipLaunchKernelGGL(slab_fill<true>, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr,
                       out_col_idx, out_g, eps_out, out_cap, sp, nrec, rec);
  else
    hipLaunchKernelGGL(slab_fill<false>, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr,
                       out_col_idx, out_g, eps_out, out_cap, sp, nrec, rec);
  const dim3 dgrid((unsigned)(p.n_itiles * p.n_slabs * p.n_chunks));
  (void)hipFuncSetAttribute((const void*)dw_slab_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);
  hipLaunchKernelGGL(dw_slab_kernel, dgrid, dim3(kDwThreads), p.lds, s, trace_in, TB, N_in, N_out, sp, rec, nrec,
                     part, p.rows_per_chunk, p.n_itiles, p.n_slabs, p.slab);
  if (p.n_chunks > 1) {
    const size_t n = (size_t)N_in * N_out;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(reduce_chunks, dim3(blocks), dim3(256), 0, s, part, p.n_chunks, n, dW);
  }
}

// Spike gradient of one layer: chunk sums, carries, the walk. share_cu keeps the walk to two
// blocks per CU so that a kernel running beside it (dW) finds room. Arguments already validated.
void enqueue_grad_in(const float* W, int T, int B, int N_in, int N_out, float alpha, const int32_t* out_row_ptr,
                     const int32_t* out_col_idx, const float* out_g, const float* eps_out, int64_t out_cap,
                     const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap, float* eps_in,
                     bool share_cu, void* workspace, hipStream_t s) {
  if (in_cap == 0) return;
  if (out_cap == 0) {  // no active output entry: delta = 0 everywhere
    fill_zero_async(eps_in, (size_t)in_cap, s);
    return;
  }
  const WalkPlan wp = plan_walk(T);
  Carve ws(workspace);
  float* Lbuf = ws.take<float>((size_t)wp.C * B * N_out);
  const int pairs = wp.C * B;
  const dim3 wgrid((pairs + kWalkWaves - 1) / kWalkWaves);
  const size_t lds = (size_t)kWalkWaves * N_out * sizeof(float);  // chunk sums only
  hipLaunchKernelGGL(gin_chunk_sums, wgrid, dim3(kWalkThreads), lds, s, T, B, N_out, alpha, wp.P, wp.C, out_row_ptr,
                     out_col_idx, out_g, eps_out, out_cap, Lbuf);
  const size_t BN = (size_t)B * N_out;
  hipLaunchKernelGGL(gin_carries, dim3((unsigned)((BN + 255) / 256)), dim3(256), 0, s, T, B, N_out, alpha, wp.P, wp.C,
                     Lbuf);
  const int nj = (N_out + kWave - 1) / kWave;
  const dim3 walk_grid(share_cu ? std::min<unsigned>(wgrid.x, 2 * kAssumedCUs) : wgrid.x);
#define SNN_WALK(NJ_)                                                                                             \
  launch_walk<NJ_>(walk_grid, 0, s, W, T, B, N_in, N_out, alpha, wp.P, wp.C, out_row_ptr, out_col_idx, out_g, eps_out, \
                   out_cap, in_row_ptr, in_col_idx, in_cap, Lbuf, eps_in)
  if (nj <= 1) SNN_WALK(1);
  else if (nj <= 2) SNN_WALK(2);
  else if (nj <= 4) SNN_WALK(4);
  else if (nj <= 8) SNN_WALK(8);
  else if (nj <= 16) SNN_WALK(16);
  else if (nj <= 32) SNN_WALK(32);
  else SNN_WALK(64);
#undef SNN_WALK
}

// common checks of the output-side CSR and its gradient
bool out_csr_ok(const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* eps_out, int64_t out_cap) {
  if (!out_row_ptr || out_cap < 0) return false;
  return out_cap == 0 || (out_col_idx && eps_out);
}

}  // namespace
}  // namespace snn

extern "C" size_t snn_sparse_dw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap) {
  if (!dims_ok(T, B, N_in, N_out) || out_cap < 0) return 0;
  return dw_workspace(T, B, N_in, N_out, out_cap);
}

extern "C" snn_status snn_sparse_dw(const float* trace_in, int T, int B, int N_in, int N_out,
                                    const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                                    const float* eps_out, int64_t out_cap, float* dW, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  if (!trace_in || !dW || !dims_ok(T, B, N_in, N_out)) return SNN_ERR_INVALID_ARG;
  if (!out_csr_ok(out_row_ptr, out_col_idx, eps_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < dw_workspace(T, B, N_in, N_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;
  enqueue_dw(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, workspace,
             static_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" size_t snn_sparse_grad_in_workspace(int T, int B, int N_out) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N_out) || too_big(T, B, N_out)) return 0;
  return gin_workspace(T, B, N_out);
}

extern "C" snn_status snn_sparse_grad_in(const float* W, int T, int B, int N_in, int N_out, float alpha,
                                         const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                                         const float* eps_out, int64_t out_cap, const int32_t* in_row_ptr,
                                         const int32_t* in_col_idx, int64_t in_cap, float* eps_in, int share_cu,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!W || !dims_ok(T, B, N_in, N_out) || bad_alpha(alpha)) return SNN_ERR_INVALID_ARG;
  if (!out_csr_ok(out_row_ptr, out_col_idx, eps_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (!in_row_ptr || in_cap < 0 || (in_cap > 0 && (!in_col_idx || !eps_in))) return SNN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < gin_workspace(T, B, N_out)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;
  enqueue_grad_in(W, T, B, N_in, N_out, alpha, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, in_row_ptr,
                  in_col_idx, in_cap, eps_in, share_cu != 0, workspace, static_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" size_t snn_sparse_backward_workspace(int T, int B, int N_in, int N_out, int64_t out_cap) {
  if (!dims_ok(T, B, N_in, N_out) || out_cap < 0) return 0;
  return align256(dw_workspace(T, B, N_in, N_out, out_cap)) + gin_workspace(T, B, N_out);
}

extern "C" snn_status snn_sparse_backward(const float* W, const float* trace_in, int T, int B, int N_in, int N_out,
                                          float alpha, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                                          const float* out_g, const float* eps_out, int64_t out_cap,
                                          const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap,
                                          float* eps_in, float* dW, void* workspace, size_t workspace_bytes,
                                          void* stream, void* aux_stream) {
  if (!W || !trace_in || !dW || !dims_ok(T, B, N_in, N_out)) return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha) || in_cap < 0) return SNN_ERR_INVALID_ARG;
  if (!out_csr_ok(out_row_ptr, out_col_idx, eps_out, out_cap)) return SNN_ERR_INVALID_ARG;
  const bool grad_in = in_row_ptr != nullptr;
  if (grad_in && in_cap > 0 && (!in_col_idx || !eps_in)) return SNN_ERR_INVALID_ARG;
  if (!grad_in && (in_col_idx || eps_in)) return SNN_ERR_INVALID_ARG;
  const size_t need = snn_sparse_backward_workspace(T, B, N_in, N_out, out_cap);
  if (!workspace || workspace_bytes < need) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* dw_ws = static_cast<char*>(workspace);
  char* gin_ws = dw_ws + align256(dw_workspace(T, B, N_in, N_out, out_cap));
  const bool do_gin = grad_in && in_cap > 0;
  // The spike gradient (L1/L2-gather bound) and dW (LDS-atomic bound) lean on different parts of
  // a CU; with an auxiliary stream they run side by side. aux waits for what is already on s,
  // and s waits for aux before anything enqueued after this call.
  hipStream_t sa = s;
  hipEvent_t ev_in = nullptr, ev_out = nullptr;
  if (do_gin && aux_stream && aux_stream != stream &&
      hipEventCreateWithFlags(&ev_in, hipEventDisableTiming) == hipSuccess &&
      hipEventCreateWithFlags(&ev_out, hipEventDisableTiming) == hipSuccess && hipEventRecord(ev_in, s) == hipSuccess &&
      hipStreamWaitEvent(static_cast<hipStream_t>(aux_stream), ev_in, 0) == hipSuccess) {
    sa = static_cast<hipStream_t>(aux_stream);
  }
  if (do_gin) {
    // beside a dW that takes longer than the walk, the walk leaves room for a dW block on every
    // CU (per product, a dW entry costs about 1.5 times a walk entry)
    const bool dw_longer = 3.0 * (double)out_cap * N_in >= 2.0 * (double)in_cap * N_out;
    enqueue_grad_in(W, T, B, N_in, N_out, alpha, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, in_row_ptr,
                    in_col_idx, in_cap, eps_in, sa != s && dw_longer, gin_ws, sa);
  }
  enqueue_dw(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, dw_ws, s);
  if (sa != s) {
    if (hipEventRecord(ev_out, sa) != hipSuccess || hipStreamWaitEvent(s, ev_out, 0) != hipSuccess)
      (void)hipStreamSynchronize(sa);  // never leave aux work unordered with later work on s
  }
  if (ev_in) (void)hipEventDestroy(ev_in);
  if (ev_out) (void)hipEventDestroy(ev_out);
  return launch_status();
}
