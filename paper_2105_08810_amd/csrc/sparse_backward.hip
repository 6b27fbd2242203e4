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
constexpr int kBufWord3 = 0x00020000;  // buffer descriptor word 3 on gfx9: 32-bit data format

struct DwPlan {
  int n_itiles, n_slabs, slab, n_chunks, rows_per_chunk;
  size_t lds;
};

DwPlan plan_dw_slab(int T, int B, int N_in, int N_out, int slab_cap) {
  DwPlan p{};
  const int TB = T * B;
  p.n_slabs = (N_out + slab_cap - 1) / slab_cap;
  p.slab = (N_out + p.n_slabs - 1) / p.n_slabs;
  p.lds = (size_t)p.slab * kLd * sizeof(double);
  p.n_itiles = (N_in + kItile - 1) / kItile;
  const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(2, (160 * 1024) / p.lds));
  const int target = cu_count() * per_cu * 8;  // short chunks: the slab blocks of a tile stay close (L2 reuse)
  const int tiles = p.n_itiles * p.n_slabs;
  int nc = (target + tiles - 1) / tiles;
  nc = std::min(nc, std::max(1, TB / (4 * N_out)));  // partial slabs stay small next to the trace
  nc = std::min(nc, 64);
  nc = std::max(nc, 1);
  p.rows_per_chunk = (TB + nc - 1) / nc;
  p.n_chunks = (TB + p.rows_per_chunk - 1) / p.rows_per_chunk;
  return p;
}

// Slabs of up to 128 outputs (one block per CU); a layer whose grid would then give fewer than
// two blocks per CU (small T B or few tiles: latency-bound, not LDS-atomic-bound) takes slabs of
// half that, two blocks per CU, twice the loads in flight.
DwPlan plan_dw(int T, int B, int N_in, int N_out) {
  const DwPlan p = plan_dw_slab(T, B, N_in, N_out, kSlab);
  if ((int64_t)p.n_itiles * p.n_slabs * p.n_chunks < 2 * cu_count()) return plan_dw_slab(T, B, N_in, N_out, kSlab / 2);
  return p;
}

// dw_slab_kernel's grid: plan_dw's slabs and input tiles, and one round of blocks over the CUs
// in chunks of interleaved row groups (about eight rounds of time-sliced chunks before: the
// last round left CUs idle and the busiest time slice set the pace; audio 700 -> 400 dW 0.099
// -> 0.089 ms, event 2312 -> 200 0.436 -> 0.383, stress at B_th 1.2 126 -> 118 ms).
DwPlan plan_dw_interleaved(int T, int B, int N_in, int N_out) {
  DwPlan p = plan_dw(T, B, N_in, N_out);
  const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(2, (160 * 1024) / p.lds));
  int nc = cu_count() * per_cu / (p.n_itiles * p.n_slabs);
  nc = std::min(nc, (T * B + kDwWaves * kRowsPerBatch - 1) / (kDwWaves * kRowsPerBatch));  // a row group each
  p.n_chunks = std::max(1, std::min(nc, 64));
  p.rows_per_chunk = 0;  // chunks take row groups round-robin
  return p;
}

// dW of layers of up to kRowsOutMax outputs and kRowsInMax inputs (dw_rows_kernel): a block
// holds all of the layer's columns for 64 inputs, so it walks the output CSR directly (no record
// passes before it); about one round of blocks over the CUs. Wider layers (two or more slabs)
// or longer input rows (more entry visits, each with its own per-entry work, at one atomic per
// visit instead of two) are faster with the slab records: a 700 -> 400 layer 0.117 against
// 0.101 ms, a 2312 -> 200 layer 0.518 against 0.447 ms; latency 784 -> 200 0.048 against
// 0.072, deep 300 -> 300 0.056 against 0.072.
constexpr int kRowsLd = kWave + 1;  // padded column of the accumulator: 64 inputs + 1
constexpr int kRowsOutMax = 300;    // 300 x 65 doubles: 156 KB of LDS
constexpr int kRowsInMax = 1024;

bool dw_rows_eligible(int N_in, int N_out) { return N_out <= kRowsOutMax && N_in <= kRowsInMax; }

DwPlan plan_dw_rows(int T, int B, int N_in, int N_out) {
  DwPlan p{};
  const int TB = T * B;
  p.n_slabs = 1;
  p.slab = N_out;
  p.lds = (size_t)N_out * kRowsLd * sizeof(double);
  p.n_itiles = (N_in + kWave - 1) / kWave;
  const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(2, (160 * 1024) / p.lds));
  int nc = cu_count() * per_cu / p.n_itiles;  // one round of blocks
  nc = std::min(nc, (TB + kDwWaves * kRowsPerBatch - 1) / (kDwWaves * kRowsPerBatch));  // a row group each at least
  p.n_chunks = std::max(1, std::min(nc, 64));
  p.rows_per_chunk = 0;  // chunks take row groups round-robin
  return p;
}

struct WalkPlan {
  int P, C;
};

WalkPlan plan_walk(int T) {
  WalkPlan w{};
  // short sequences: chunks of two steps (T = 100: 50 chunks; deep's spike gradients 0.036-0.047
  // -> 0.031-0.042 ms, the walks being latency-bound); longer ones: T / 32 steps (stress, T = 500:
  // 16; 8 made it slower, the chunk sums and carries growing with the chunk count)
  w.P = T <= 128 ? 2 : std::min(64, (T + 31) / 32);
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
                                                             float* __restrict__ out, int n_chunks,
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

  // Chunk c takes the groups of kDwWaves * kRowsPerBatch rows c, c + n_chunks, ...: every chunk
  // spans the whole time axis, so that one round of blocks finishes together wherever the
  // activity lies in time. Wavefront w takes rows [8 w, 8 w + 8) of each of its chunk's groups.
  const int r_hi = TB;
  const int2* rec2 = reinterpret_cast<const int2*>(rec);
  // Software pipeline over batches of 8 rows: while a batch is processed, the next batch's
  // trace values and records are in flight and the row pointers of the one after it. Rows past
  // TB read sp[TB] (empty ranges); a row with no entry in this slab reads the batch's first
  // trace row instead of its own (a cache hit, never used).
  auto load_sp = [&](int rb) { return spl[min(rb + min(l, kRowsPerBatch), r_hi)]; };
  auto load_rest = [&](int rb, int spv, float* t0, float* t1, int2& ra) {
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      const bool any = rdlane(spv, k + 1) > rdlane(spv, k);
      const size_t row = (size_t)(any ? min(rb + k, r_hi - 1) : min(rb, r_hi - 1)) * N_in;
      t0[k] = trace[row + ic0];
      t1[k] = trace[row + ic1];
    }
    ra = rec2[min((int64_t)rdlane(spv, 0) + l, nrec - 1)];  // lane s holds the batch's record s
  };
  const int kStride = kDwWaves * kRowsPerBatch * n_chunks;
  int rb = c * kDwWaves * kRowsPerBatch + w * kRowsPerBatch;
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
  for (int ii = w; ii < kItile && it * kItile + ii < N_in; ii += kDwWaves)  // a wavefront per input row
    for (int jj = l; jj < width; jj += kWave)
      dst[(size_t)(it * kItile + ii) * N_out + j0 + jj] = (float)acc[jj * kLd + ii];
}

// Block (c, it) of dw_rows: inputs [64 it, 64 it + 64) (one per lane), every output, the rows of
// chunk c, read straight from the output CSR: G = eps g is formed from the entries (the product
// slab_fill stores); entries whose column is outside [0, N_out) are skipped. Each wavefront takes
// kRowsPerBatch rows at a time, their trace values and first 64 entries in flight while the
// previous batch is added into the float64 accumulators (one LDS atomic per entry: lanes are
// inputs); a batch of more than 64 entries loads the rest 64 at a time. The trace slice of a
// (row, input tile) is read once.
template <bool HAS_G>
__global__ __launch_bounds__(kDwThreads) void dw_rows_kernel(const float* __restrict__ trace, int TB, int N_in,
                                                             int N_out, const int32_t* __restrict__ row_ptr,
                                                             const int32_t* __restrict__ col_idx,
                                                             const float* __restrict__ g,
                                                             const float* __restrict__ eps, int64_t cap,
                                                             float* __restrict__ out, int n_chunks,
                                                             int n_itiles) {
  extern __shared__ double acc[];  // [N_out][kRowsLd]
  int id = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) id = (id & 7) * (nb >> 3) + (id >> 3);
  const int c = id / n_itiles;
  const int it = id - c * n_itiles;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int ic = min(it * kWave + l, N_in - 1);  // lanes past N_in accumulate rows that are never written out
  char* accb = reinterpret_cast<char*>(acc) + l * (int)sizeof(double);

  for (int k = tid; k < N_out * kRowsLd; k += kDwThreads) acc[k] = 0.0;
  __syncthreads();

  // Chunk c takes the groups of kGroup = 128 rows c, c + n_chunks, c + 2 n_chunks, ...: every
  // chunk spans the whole time axis, so that chunks get about as many entries wherever the
  // activity lies in time. Wavefront w takes rows [8 w, 8 w + 8) of each of its chunk's groups.
  // lane k <= kRowsPerBatch: row pointer rb + k (rows past TB read TB's: empty ranges)
  auto load_rp = [&](int rb) { return clamp_entry(row_ptr[min(rb + min(l, kRowsPerBatch), TB)], cap); };
  // the batch's trace values (a row with no entry reads the batch's first row instead: a cache
  // hit, never used) and, in lane s, its entry s (lanes past the entries read a valid one). G is
  // formed only when the batch is added in, so that issuing these loads waits for none of them.
  auto load_rest = [&](int rpv, int rb, float* t, int& col, float& ep, float& gg) {
    const int r0 = min(rb, TB - 1);
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      const bool any = rdlane(rpv, k + 1) > rdlane(rpv, k);
      t[k] = trace[(size_t)(any ? min(rb + k, TB - 1) : r0) * N_in + ic];
    }
    const int E0 = rdlane(rpv, 0);
    const int E1 = rdlane(rpv, kRowsPerBatch);
    const int64_t q = std::max<int64_t>(0, std::min<int64_t>(min(E0 + l, E1 - 1), cap - 1));
    col = col_idx[q];
    ep = eps[q];
    gg = HAS_G ? g[q] : 1.0f;
  };
  constexpr int kGroup = kDwWaves * kRowsPerBatch;
  const int stride = kGroup * n_chunks;
  int rb = c * kGroup + w * kRowsPerBatch;
  int rpv = load_rp(rb);
  float tr[kRowsPerBatch];
  int col;
  float ep, gg;
  load_rest(rpv, rb, tr, col, ep, gg);
  int rpv_n = load_rp(rb + stride);
  for (; rb < TB; rb += stride) {
    float tn[kRowsPerBatch];
    int col_n;
    float ep_n, gg_n;
    load_rest(rpv_n, rb + stride, tn, col_n, ep_n, gg_n);
    const int rpv_nn = load_rp(rb + 2 * stride);
    __builtin_amdgcn_sched_barrier(0);
    // the batch's first 64 entries from (col, G), loaded with the trace values; the rest of a
    // batch of more than 64 (rare) in a second pass, 64 per coalesced load. Kept apart so that
    // the first pass waits only for this batch's loads, not for the next batch's.
    const float G = ep * gg;
    const int base = rdlane(rpv, 0);
    const int e_end = rdlane(rpv, kRowsPerBatch);
    const int e_reg = min(e_end, base + kWave);
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      const double t = (double)tr[k];
      const int lo = rdlane(rpv, k);
      const int hi = min(rdlane(rpv, k + 1), e_reg);
      for (int e = lo; e < hi; ++e) {
        const int j = rdlane(col, e - base);
        if ((unsigned)j < (unsigned)N_out) {
          double* a = reinterpret_cast<double*>(accb + j * kRowsLd * (int)sizeof(double));
          atomicAdd(a, t * (double)rdlane(G, e - base));
        }
      }
    }
    for (int pb = base + kWave; pb < e_end; pb += kWave) {
      const int64_t q = std::min<int64_t>(min(pb + l, e_end - 1), cap - 1);  // e_end <= cap
      const int colp = col_idx[q];
      const float Gp = eps[q] * (HAS_G ? g[q] : 1.0f);
      const int pe = min(e_end, pb + kWave);
#pragma unroll
      for (int k = 0; k < kRowsPerBatch; ++k) {
        const double t = (double)tr[k];
        const int lo = max(rdlane(rpv, k), pb);
        const int hi = min(rdlane(rpv, k + 1), pe);
        for (int e = lo; e < hi; ++e) {
          const int j = rdlane(colp, e - pb);
          if ((unsigned)j < (unsigned)N_out) {
            double* a = reinterpret_cast<double*>(accb + j * kRowsLd * (int)sizeof(double));
            atomicAdd(a, t * (double)rdlane(Gp, e - pb));
          }
        }
      }
    }
    rpv = rpv_n;
    rpv_n = rpv_nn;
    col = col_n;
    ep = ep_n;
    gg = gg_n;
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) tr[k] = tn[k];
  }
  __syncthreads();
  float* dst = out + (size_t)c * N_in * N_out;
  for (int ii = w; ii < kWave && it * kWave + ii < N_in; ii += kDwWaves)  // a wavefront per input row
    for (int jj = l; jj < N_out; jj += kWave) dst[(size_t)(it * kWave + ii) * N_out + jj] = (float)acc[jj * kRowsLd + ii];
}

// dW with the input trace rebuilt from the input spikes (trace recompute). The trace at every
// K-th step (checkpoints) and the spikes S_in replace the stored trace: the trace recurrence runs
// forward in registers with the float32 operations of the forward, so every trace value equals
// the stored one bit for bit. Block = (chunk: steps [t_lo, t_lo + tlen) x 128 samples, input
// tile, slab). Wavefront w owns 8 samples and walks the chunk's steps; at step t its batch is the
// rows t B + b of its samples, with their trace values in the lane's registers (8 samples x 2
// inputs); after the batch the registers advance one step with S[t]. Records, LDS accumulators,
// the per-entry work and the software pipeline (the next step's records, row pointers and spikes
// in flight) are those of dw_slab_kernel.
constexpr int kSamplesPerChunk = kDwWaves * kRowsPerBatch;

__global__ __launch_bounds__(kDwThreads) void dw_slab_spikes_kernel(
    const uint8_t* __restrict__ s_in, const float* __restrict__ ck, int K, float alpha, int T, int B, int N_in,
    int N_out, const int32_t* __restrict__ sp, const SlabRec* __restrict__ rec, int64_t nrec, float* __restrict__ out,
    int tlen, int n_bblk, int n_itiles, int n_slabs, int slab) {
#pragma clang fp contract(off)  // the trace recurrence rounds its product and its sum separately
  extern __shared__ double acc[];  // [slab][kLd]
  int id = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) id = (id & 7) * (nb >> 3) + (id >> 3);
  const int tiles = n_itiles * n_slabs;
  const int c = id / tiles;
  const int sl = (id - c * tiles) % n_slabs;
  const int it = (id - c * tiles) / n_slabs;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int TB = T * B;
  const int i0 = it * kItile + l;
  const int ic0 = min(i0, N_in - 1);
  const int ic1 = min(i0 + kWave, N_in - 1);
  const int j0 = sl * slab;
  const int j1 = min(N_out, j0 + slab);
  const int32_t* spl = sp + (size_t)sl * TB;
  char* accb = reinterpret_cast<char*>(acc) + l * (int)sizeof(double);
  const int max_off = (slab - 1) * kLd * (int)sizeof(double);

  for (int k = tid; k < slab * kLd; k += kDwThreads) acc[k] = 0.0;
  __syncthreads();

  const int tb = c / n_bblk;
  const int bb = c - tb * n_bblk;
  const int t_lo = tb * tlen;  // a multiple of K
  const int t_hi = min(T, t_lo + tlen);
  const int b0 = bb * kSamplesPerChunk + w * kRowsPerBatch;
  const int nbv = max(0, min(kRowsPerBatch, B - b0));  // this wavefront's samples
  const int2* rec2 = reinterpret_cast<const int2*>(rec);
  float tr0[kRowsPerBatch], tr1[kRowsPerBatch];
#pragma unroll
  for (int k = 0; k < kRowsPerBatch; ++k) {
    const size_t row = ((size_t)(t_lo / K) * B + min(b0 + k, B - 1)) * N_in;
    tr0[k] = ck[row + ic0];
    tr1[k] = ck[row + ic1];
  }
  // lane k <= 8: row pointer of row t B + b0 + min(k, nbv) (rows past the samples: empty ranges)
  auto load_sp = [&](int t) { return spl[(size_t)t * B + min(b0, B - 1) + min(l, nbv)]; };
  auto load_rec = [&](int spv) { return rec2[min((int64_t)rdlane(spv, 0) + l, nrec - 1)]; };
  auto load_spk = [&](int t, uint32_t* sk) {  // S[t] of the 8 samples at the lane's two inputs
#pragma unroll
    for (int k = 0; k < kRowsPerBatch; ++k) {
      const uint8_t* row = s_in + ((size_t)t * B + min(b0 + k, B - 1)) * N_in;
      sk[k] = (uint32_t)row[ic0] | ((uint32_t)row[ic1] << 8);
    }
  };
  if (nbv > 0 && t_lo < t_hi) {
    int spv = load_sp(t_lo);
    int2 ra = load_rec(spv);
    uint32_t sk[kRowsPerBatch];
    load_spk(t_lo, sk);
    int spv_n = load_sp(min(t_lo + 1, T - 1));
    for (int t = t_lo; t < t_hi; ++t) {
      const int2 ran = load_rec(spv_n);
      uint32_t skn[kRowsPerBatch];
      load_spk(min(t + 1, T - 1), skn);
      const int spv_nn = load_sp(min(t + 2, T - 1));
      __builtin_amdgcn_sched_barrier(0);
      const int base = rdlane(spv, 0);
      const int n = rdlane(spv, kRowsPerBatch) - base;
      if (n <= kWave) {
        int lo = 0;
#pragma unroll
        for (int k = 0; k < kRowsPerBatch; ++k) {
          const double t0 = (double)tr0[k], t1 = (double)tr1[k];
          const int hi = rdlane(spv, k + 1) - base;
          for (int s = lo; s < hi; ++s) {
            const int off = (int)min((unsigned)rdlane(ra.x, s), (unsigned)max_off);
            const double G = (double)__int_as_float(rdlane(ra.y, s));
            double* a = reinterpret_cast<double*>(accb + off);
            atomicAdd(a, t0 * G);
            atomicAdd(a + kWave, t1 * G);
          }
          lo = hi;
        }
      } else {
#pragma unroll
        for (int k = 0; k < kRowsPerBatch; ++k) {
          const double t0 = (double)tr0[k], t1 = (double)tr1[k];
          const int lo = rdlane(spv, k);
          const int hi = rdlane(spv, k + 1);
          for (int s = lo; s < hi; ++s) {
            const int2 x = rec2[min((int64_t)s, nrec - 1)];
            const double G = (double)__int_as_float(x.y);
            double* a = reinterpret_cast<double*>(accb + min(max(x.x, 0), max_off));
            atomicAdd(a, t0 * G);
            atomicAdd(a + kWave, t1 * G);
          }
        }
      }
      // trace[t + 1] = alpha trace[t] + S[t], separately rounded as in the forward
#pragma unroll
      for (int k = 0; k < kRowsPerBatch; ++k) {
        tr0[k] = alpha * tr0[k] + ((sk[k] & 0xffu) ? 1.0f : 0.0f);  // not fused (contract off)
        tr1[k] = alpha * tr1[k] + ((sk[k] & 0xff00u) ? 1.0f : 0.0f);
        sk[k] = skn[k];
      }
      spv = spv_n;
      spv_n = spv_nn;
      ra = ran;
    }
  }
  __syncthreads();
  float* dst = out + (size_t)c * N_in * N_out;
  const int width = j1 - j0;
  for (int ii = w; ii < kItile && it * kItile + ii < N_in; ii += kDwWaves)  // a wavefront per input row
    for (int jj = l; jj < width; jj += kWave)
      dst[(size_t)(it * kItile + ii) * N_out + j0 + jj] = (float)acc[jj * kLd + ii];
}

// Trace checkpoints: ck[q, b, i] = the input trace at step q K (q < ceil(T / K)), from the spikes
// by the forward's recurrence (one thread per (b, i)).
__global__ void trace_checkpoints_kernel(const uint8_t* __restrict__ s_in, int T, int B, int N_in, float alpha, int K,
                                         float* __restrict__ ck) {
#pragma clang fp contract(off)  // the trace recurrence rounds its product and its sum separately
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // b * N_in + i
  if (k >= (int64_t)B * N_in) return;
  const int64_t step = (int64_t)B * N_in;
  float tr = 0.0f;
  for (int t0 = 0; t0 < T; t0 += K) {
    ck[(int64_t)(t0 / K) * step + k] = tr;
    const int t1 = min(T - 1, t0 + K);  // advance to step t1 (or stop at the last step)
    uint8_t sv[16];
    for (int t = t0; t < t1; t += 16) {
      const int m = min(16, t1 - t);
#pragma unroll
      for (int u = 0; u < 16; ++u) sv[u] = s_in[(int64_t)(t + min(u, m - 1)) * step + k];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (u < m) tr = alpha * tr + (sv[u] ? 1.0f : 0.0f);  // not fused (contract off)
    }
  }
}

__global__ void fill_zero(float* __restrict__ p, size_t n) {
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) p[k] = 0.0f;
}

__global__ void reduce_chunks(const float* __restrict__ part, int n_chunks, size_t n, float* __restrict__ out) {
  constexpr int kAhead = 8;  // partials loaded before any is added (the adds keep chunk order)
  for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    double s = 0.0;  // fixed order, rounded once
    int c = 0;
    for (; c + kAhead <= n_chunks; c += kAhead) {
      float v[kAhead];
#pragma unroll
      for (int u = 0; u < kAhead; ++u) v[u] = part[(size_t)(c + u) * n + k];
#pragma unroll
      for (int u = 0; u < kAhead; ++u) s += (double)v[u];
    }
    for (; c < n_chunks; ++c) s += (double)part[(size_t)c * n + k];
    out[k] = (float)s;
  }
}

// ------------------------------------------------------------------ narrow layers
//
// With few outputs (N_out <= kNarrowOut, e.g. a readout of a few classes) a wavefront per row
// or per (chunk, sample) wastes most lanes. Narrow layers work from G written densely instead,
// rows padded to ld = 8, 16 or 32 columns (zeros past N_out), so that a row is one uniform
// load:
//   spike gradient: delta for every (t, b, j) by one thread per (b, j) walking t down, then one
//     lane per input-active entry forms W[i, :] . delta[t, b, :] (ascending j);
//   dW: a wavefront owns 64 inputs, 8 or 16 columns and a chunk of rows, visits the rows that
//     have an entry (a bitset of them is built once) eight at a time and keeps sums per (input,
//     column) (float32 over 64 rows, then float64); one float partial per chunk, summed in chunk
//     order.
// Deterministic.
constexpr int kNarrowOut = 32;
static_assert(kNarrowOut <= kWave, "one lane per output column in the G scatter");
constexpr int kNarrowBatch = 8;  // 8 rows x 8 (or more) columns fill at least one load of 64 lanes

int narrow_ld(int N_out) { return N_out <= 8 ? 8 : (N_out <= 16 ? 16 : 32); }

// One wave per row writes the row's whole padded G: lane j < ld owns column j and picks its
// value out of the row's entries, which the wave reads 64 at a time.
__global__ void narrow_scatter_g(int TB, int N_out, int ld, const int32_t* __restrict__ rp,
                                 const int32_t* __restrict__ col, const float* __restrict__ g,
                                 const float* __restrict__ eps, int64_t cap, float* __restrict__ Gd) {
  const int r = __builtin_amdgcn_readfirstlane((int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave));
  if (r >= TB) return;
  const int l = lane_id();
  const int64_t e0 = clamp_entry(rp[r], cap);
  const int64_t e1 = clamp_entry(rp[r + 1], cap);
  float x = 0.0f;
  for (int64_t base = e0; base < e1; base += kWave) {
    const int64_t e = base + l;
    int c = -1;
    float v = 0.0f;
    if (e < e1) {
      c = col[e];
      v = g ? eps[e] * g[e] : eps[e];
    }
    const int n = (int)std::min<int64_t>(e1 - base, kWave);
    for (int k = 0; k < n; ++k) {
      const int ck = __shfl(c, k);
      const float vk = __shfl(v, k);
      if (ck == l && l < N_out) x = vk;
    }
  }
  if (l < ld) Gd[(int64_t)r * ld + l] = x;
}

// D[T-1] = 0, D[t] = alpha D[t+1] + G[t+1] for each (b, column); BL = B * ld. The G values of
// 32 steps are loaded at once (the recurrence waits only on its own multiply-add).
constexpr int kDeltaSteps = 32;

__global__ void narrow_delta(int T, int64_t BL, float alpha, const float* __restrict__ Gd, float* __restrict__ D) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= BL) return;
  float d = 0.0f;
  D[(int64_t)(T - 1) * BL + k] = 0.0f;
  for (int t1 = T - 1; t1 > 0; t1 -= kDeltaSteps) {  // steps t = t1 - 1 down to t1 - 32 (>= 0)
    float g[kDeltaSteps];
#pragma unroll
    for (int u = 0; u < kDeltaSteps; ++u) g[u] = t1 - u >= 1 ? Gd[(int64_t)(t1 - u) * BL + k] : 0.0f;
#pragma unroll
    for (int u = 0; u < kDeltaSteps; ++u) {
      if (t1 - u >= 1) {
        d = alpha * d + g[u];
        D[(int64_t)(t1 - u - 1) * BL + k] = d;
      }
    }
  }
}

// eps_in at each input-active entry of row r = t B + b: W[i, :] . D[r, :]; the padded columns of
// D are zero, so the weight index is clamped to the row instead of tested.
template <int NJ>
__global__ void narrow_gin(int TB, int N_in, int N_out, const float* __restrict__ W, const float* __restrict__ D,
                           const int32_t* __restrict__ rp, const int32_t* __restrict__ col, int64_t cap,
                           float* __restrict__ eps_in) {
  const int r = __builtin_amdgcn_readfirstlane((int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave));
  if (r >= TB) return;
  const int64_t e0 = clamp_entry(rp[r], cap);
  const int64_t e1 = clamp_entry(rp[r + 1], cap);
  if (e0 >= e1) return;
  const float* d = D + (int64_t)r * NJ;
  float dv[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) dv[j] = d[j];
  for (int64_t e = e0 + lane_id(); e < e1; e += kWave) {
    const int i = col[e];
    const int ic = min(max(i, 0), N_in - 1);
    const float* w = W + (int64_t)ic * N_out;
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) s += w[min(j, N_out - 1)] * dv[j];
    eps_in[e] = (unsigned)i < (unsigned)N_in ? s : 0.0f;
  }
}

// Bit k of word w: row 64 w + k has an entry.
__global__ void narrow_busy_rows(int TB, const int32_t* __restrict__ rp, int64_t cap, uint64_t* __restrict__ busy) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  const bool on = r < TB && clamp_entry(rp[r + 1], cap) > clamp_entry(rp[r], cap);
  const uint64_t m = __ballot(on);
  if (lane_id() == 0 && r < TB) busy[r / kWave] = m;
}

struct NarrowDwPlan {
  int n_iw, n_chunks, rows_per_chunk;  // rows_per_chunk: a multiple of 8
};

NarrowDwPlan plan_narrow_dw(int T, int B, int N_in) {
  NarrowDwPlan p{};
  const int TB = T * B;
  p.n_iw = (N_in + kWave - 1) / kWave;
  constexpr int kMaxRows = 63 * kWave;  // a chunk (starting at a multiple of 8) spans <= 64 bitset words
  const int units = (TB + kNarrowBatch - 1) / kNarrowBatch;
  int nc = (32 * cu_count() + p.n_iw - 1) / p.n_iw;  // about 32 wavefronts per CU
  nc = std::min(nc, std::min(units, 1024));
  nc = std::max(nc, (TB + kMaxRows - 1) / kMaxRows);
  p.rows_per_chunk = std::min(kMaxRows, ((units + nc - 1) / nc) * kNarrowBatch);
  p.n_chunks = (TB + p.rows_per_chunk - 1) / p.rows_per_chunk;
  return p;
}

template <int NJ>
__global__ void narrow_dw(const float* __restrict__ trace, int TB, int N_in, int N_out,
                          const uint64_t* __restrict__ busy, const float* __restrict__ Gd, int ld, int rows_per_chunk,
                          int n_iw, float* __restrict__ part) {
  const int j0 = blockIdx.y * NJ;  // this block's columns: j0 .. j0 + NJ - 1 of the padded G
  const int wv = __builtin_amdgcn_readfirstlane((int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave));
  const int c = wv / n_iw;
  const int iw = wv - c * n_iw;
  const int r_lo = c * rows_per_chunk;
  if (r_lo >= TB) return;
  const int r_hi = min(TB, r_lo + rows_per_chunk);
  const int l = lane_id();
  const int i = iw * kWave + l;
  const int ic = min(i, N_in - 1);  // lanes past N_in read a valid column and write nothing
  // float32 sums over up to 64 rows (eight batches), added into float64 sums: the rounding error
  // stays at the level of a 64-term float32 sum, at float32 arithmetic's speed
  double acc[NJ];
  float acc32[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    acc[j] = 0.0;
    acc32[j] = 0.0f;
  }
  int pending = 0;
  auto flush = [&]() {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      acc[j] += (double)acc32[j];
      acc32[j] = 0.0f;
    }
    pending = 0;
  };
  const int w_lo = r_lo / kWave;
  const int nw = (r_hi + kWave - 1) / kWave - w_lo;  // at most 64 bitset words (the plan's chunks)
  uint64_t mine = l < nw ? busy[w_lo + l] : 0ull;
  if (l == 0) mine &= ~0ull << (r_lo & (kWave - 1));  // rows of the chunk only
  if (l == nw - 1 && (r_hi & (kWave - 1))) mine &= (1ull << (r_hi & (kWave - 1))) - 1;
  auto word = [&](int q) {  // uniform: the rows' G loads become scalar-indexed
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(mine >> 32), q) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mine, q);
  };
  int q = 0;
  uint64_t m = word(0);
  // the next (up to) eight rows with an entry; rows past the count are r_lo (loaded, weight 0)
  auto next_rows = [&](int* rows) {
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < kNarrowBatch; ++k) {
      while (m == 0 && q + 1 < nw) m = word(++q);
      rows[k] = m ? (w_lo + q) * kWave + (int)__builtin_ctzll(m) : r_lo;
      cnt += m ? 1 : 0;
      m &= m - 1;
    }
    return cnt;
  };
  // A batch's G rows (8 x NJ values) spread over the lanes, NJ / 8 per lane, and its trace values;
  // a G value is broadcast by a lane read when it is used.
  constexpr int kSlots = NJ * kNarrowBatch / kWave;
  auto load = [&](const int* rows, float* tv, float* gv) {
    int rowv = rows[0];
#pragma unroll
    for (int k = 1; k < kNarrowBatch; ++k) rowv = l == k ? rows[k] : rowv;
#pragma unroll
    for (int z = 0; z < kSlots; ++z) {
      const int f = z * kWave + l;
      gv[z] = Gd[(int64_t)__shfl(rowv, f / NJ) * ld + j0 + (f % NJ)];
    }
#pragma unroll
    for (int k = 0; k < kNarrowBatch; ++k) tv[k] = trace[(int64_t)rows[k] * N_in + ic];
  };
  auto accumulate = [&](const float* tv, const float* gv, int cnt) {
#pragma unroll
    for (int k = 0; k < kNarrowBatch; ++k) {
      const float t = k < cnt ? tv[k] : 0.0f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int f = k * NJ + j;
        const float g = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gv[f / kWave]), f % kWave));
        acc32[j] = fmaf(t, g, acc32[j]);
      }
    }
    if (++pending == kNarrowBatch) flush();
  };
  // two batches in flight: the next one's loads are issued before this one's sums (ping-pong
  // between two register sets, so no loaded value is copied)
  int ra[kNarrowBatch], rn[kNarrowBatch];
  float ta[kNarrowBatch], tn[kNarrowBatch], ga[kSlots], gn[kSlots];
  int ca = next_rows(ra);
  if (ca > 0) {
    load(ra, ta, ga);
    while (true) {
      const int cn = next_rows(rn);
      load(rn, tn, gn);
      accumulate(ta, ga, ca);
      if (cn == 0) break;
      ca = next_rows(ra);
      load(ra, ta, ga);
      accumulate(tn, gn, cn);
      if (ca == 0) break;
    }
  }
  flush();
  if (i < N_in) {
    float* dst = part + ((int64_t)c * N_in + i) * N_out;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j0 + j < N_out) dst[j0 + j] = (float)acc[j];
  }
}

// dW = sum of the chunk partials: a block of 16 wavefronts per 64 outputs, wavefront w summing
// chunks w, w + 16, ... in order, then the 16 sums in order (float64 throughout).
constexpr int kReduceWaves = 16;

__global__ __launch_bounds__(kReduceWaves * kWave) void narrow_reduce(const float* __restrict__ part, int n_chunks,
                                                                      int64_t n, float* __restrict__ out) {
  __shared__ double red[kReduceWaves][kWave];
  const int l = lane_id();
  const int w = threadIdx.x / kWave;
  const int64_t k = (int64_t)blockIdx.x * kWave + l;
  double s = 0.0;
  if (k < n) {
#pragma unroll 4
    for (int c = w; c < n_chunks; c += kReduceWaves) s += (double)part[(int64_t)c * n + k];
  }
  red[w][l] = s;
  __syncthreads();
  if (w == 0 && k < n) {
    double t = 0.0;
#pragma unroll
    for (int v = 0; v < kReduceWaves; ++v) t += red[v][l];
    out[k] = (float)t;
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
  constexpr int kAhead = 8;  // chunk sums loaded before the carries overwrite them
  int c = C - 1;
  for (; c + 1 >= kAhead; c -= kAhead) {
    float Lv[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) Lv[u] = buf[(size_t)(c - u) * BN + k];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      buf[(size_t)(c - u) * BN + k] = x;
      x = (c - u == C - 1 ? aLast : aP) * x + Lv[u];
    }
  }
  for (; c >= 0; --c) {
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

// The walk for layers whose outputs are a multiple of 4 (and more than 256): lane l holds
// delta at j = 4 l + 256 m + u (u < 4), so a W row arrives in 16-byte loads, NJ / 4 per lane.
// G[t] goes into delta through a per-wavefront LDS row: the step's output entries are stored
// at their columns (one lane each, no two alike inside a row), every lane then takes its
// columns with 16-byte reads (delta <- alpha delta + G) and the entries' columns are cleared
// again. This replaces a register-indexed add per output entry.
template <int NJ>
__global__ __launch_bounds__(kWalkThreads, NJ <= 16 ? 4 : 1) void gin_walk_x4(
    const float* __restrict__ W, int T, int B, int N_in, int N_out, float alpha, int P, int C,
    const int32_t* __restrict__ orp, const int32_t* __restrict__ oci, const float* __restrict__ og,
    const float* __restrict__ oeps, int64_t ocap, const int32_t* __restrict__ irp,
    const int32_t* __restrict__ ici, int64_t icap, const float* __restrict__ D, float* __restrict__ eps_in) {
  static_assert(NJ % 4 == 0, "whole 16-byte columns per lane");
  constexpr int NQ = NJ / 4;
  extern __shared__ float4 gq_all[];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  float4* gq = gq_all + (size_t)w * NQ * kWave;  // the wavefront's G row: column j at float j
  float* gcol = reinterpret_cast<float*>(gq);
#pragma unroll
  for (int m = 0; m < NQ; ++m) gq[l + kWave * m] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int q = blockIdx.x * kWalkWaves + w; q < C * B; q += gridDim.x * kWalkWaves) {
    const int c = q / B;
    const int b = q - c * B;
    float d[NJ];
#pragma unroll
    for (int m = 0; m < NQ; ++m) {
      const int j = 4 * l + 4 * kWave * m;
      const float4 v = j < N_out ? *reinterpret_cast<const float4*>(D + (size_t)q * N_out + j)
                                 : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      d[4 * m + 0] = v.x;
      d[4 * m + 1] = v.y;
      d[4 * m + 2] = v.z;
      d[4 * m + 3] = v.w;
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
    // entry l of step k's rows (clamped into the row; only lanes below the row length are used)
    auto in_idx = [&](int k) {
      const int a = rdlane(ia, k), z = rdlane(ib, k);
      return z > a ? ici[min(a + l, z - 1)] : -1;
    };
    auto out_col = [&](int k) {
      const int a = rdlane(oa, k), z = rdlane(ob, k);
      return z > a ? oci[min(a + l, z - 1)] : -1;
    };
    // eps and g of entry l of step k's output row, multiplied where they are used (a product here
    // would wait for the loads at once)
    auto out_e = [&](int k) {
      const int a = rdlane(oa, k), z = rdlane(ob, k);
      return z > a ? oeps[min(a + l, z - 1)] : 0.0f;
    };
    auto out_gg = [&](int k) {
      const int a = rdlane(oa, k), z = rdlane(ob, k);
      return (z > a && og) ? og[min(a + l, z - 1)] : 1.0f;
    };
    int k = t_hi - 1 - t_lo;
    int vi = in_idx(k), vj = out_col(k);
    float ve = out_e(k), vgg = out_gg(k);
    for (; k >= 0; --k) {
      // eps_in at the input-active entries of row (t, b), with delta[t] = d
      const int i0 = rdlane(ia, k);
      const int i1 = rdlane(ib, k);
      // This step's entries are copied out of the registers the next step's requests go to, and
      // the first batch's inputs read, before those requests: vector memory counts retire in order,
      // so a later read of these registers would wait for the new requests too.
      int iv0[kGinBatch];
#pragma unroll
      for (int u = 0; u < kGinBatch; ++u) {
        const int xi = rdlane(vi, u);
        iv0[u] = (u < i1 - i0 && (unsigned)xi < (unsigned)N_in) ? xi : -1;
      }
      int vc = vi;  // entry i0 + l
      const int vj_k = vj;
      const float vg_k = ve * vgg;
      const int kn = max(k - 1, 0);
      vi = in_idx(kn);
      vj = out_col(kn);
      ve = out_e(kn);
      vgg = out_gg(kn);
      for (int e0 = i0; e0 < i1; e0 += kWave) {
        if (e0 > i0) vc = ici[min(e0 + l, i1 - 1)];  // entry e0 + l
        const int ne = min(kWave, i1 - e0);
        for (int x = 0; x < ne; x += kGinBatch) {
          int iv[kGinBatch];
          if (e0 == i0 && x == 0) {
#pragma unroll
            for (int u = 0; u < kGinBatch; ++u) iv[u] = iv0[u];
          } else {
#pragma unroll
            for (int u = 0; u < kGinBatch; ++u) {
              const int xi = rdlane(vc, min(x + u, kWave - 1));
              iv[u] = (x + u < ne && (unsigned)xi < (unsigned)N_in) ? xi : -1;
            }
          }
          float wv[kGinBatch][NJ];
#pragma unroll
          for (int u = 0; u < kGinBatch; ++u) {
            const __amdgpu_buffer_rsrc_t rs = row_rsrc(W + (size_t)(iv[u] >= 0 ? iv[u] : 0) * N_out, N_out);
#pragma unroll
            for (int m = 0; m < NQ; ++m) {
              const auto v4 = __builtin_amdgcn_raw_buffer_load_b128(rs, (4 * l + 4 * kWave * m) * 4, 0, 0);
              wv[u][4 * m + 0] = __uint_as_float(v4[0]);
              wv[u][4 * m + 1] = __uint_as_float(v4[1]);
              wv[u][4 * m + 2] = __uint_as_float(v4[2]);
              wv[u][4 * m + 3] = __uint_as_float(v4[3]);
            }
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
          if ((l & 15) == 0 && x + u < ne) eps_in[e0 + x + u] = tot;
        }
      }
      // delta[t-1] = alpha delta[t] + G[t], G through the LDS row
      const int o0 = rdlane(oa, k);
      const int o1 = rdlane(ob, k);
      for (int e0 = o0; e0 < o1; e0 += kWave) {
        int jv = vj_k;
        float gv = vg_k;
        if (e0 > o0) {  // rows with more than 64 active outputs: the rest is read here
          const int ec = min(e0 + l, o1 - 1);
          jv = oci[ec];
          gv = oeps[ec] * (og ? og[ec] : 1.0f);
        }
        if (e0 + l < o1 && (unsigned)jv < (unsigned)N_out) gcol[jv] = gv;
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int m = 0; m < NQ; ++m) {
        const float4 g4 = gq[l + kWave * m];
        d[4 * m + 0] = alpha * d[4 * m + 0] + g4.x;
        d[4 * m + 1] = alpha * d[4 * m + 1] + g4.y;
        d[4 * m + 2] = alpha * d[4 * m + 2] + g4.z;
        d[4 * m + 3] = alpha * d[4 * m + 3] + g4.w;
      }
      __builtin_amdgcn_wave_barrier();
      if (o1 - o0 <= kWave) {
        if (o0 + l < o1 && (unsigned)vj_k < (unsigned)N_out) gcol[vj_k] = 0.0f;
      } else {
#pragma unroll
        for (int m = 0; m < NQ; ++m) gq[l + kWave * m] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

template <int NJ>
void launch_walk_x4(dim3 grid, hipStream_t s, const float* W, int T, int B, int N_in, int N_out, float alpha, int P,
                    int C, const int32_t* orp, const int32_t* oci, const float* og, const float* oeps, int64_t ocap,
                    const int32_t* irp, const int32_t* ici, int64_t icap, const float* D, float* eps_in) {
  const size_t lds = (size_t)kWalkWaves * NJ * kWave * sizeof(float);
  hipLaunchKernelGGL(gin_walk_x4<NJ>, grid, dim3(kWalkThreads), lds, s, W, T, B, N_in, N_out, alpha, P, C, orp, oci,
                     og, oeps, ocap, irp, ici, icap, D, eps_in);
}

}  // namespace
}  // namespace snn

using namespace snn;

namespace snn {
namespace {

size_t dw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap) {
  if (N_out <= kNarrowOut) {  // padded dense G, the busy-row bitset and the chunk partials
    const NarrowDwPlan q = plan_narrow_dw(T, B, N_in);
    Carve c(nullptr);
    c.take<float>((size_t)T * B * narrow_ld(N_out));
    c.take<uint64_t>(((size_t)T * B + kWave - 1) / kWave);
    if (q.n_chunks > 1) c.take<float>((size_t)q.n_chunks * N_in * N_out);
    return c.off;
  }
  if (mdw_eligible(T, B, N_in, N_out, out_cap)) return mdw_workspace(T, B, N_in, N_out, out_cap);
  if (dw_rows_eligible(N_in, N_out)) {  // the chunk partials only
    const DwPlan p = plan_dw_rows(T, B, N_in, N_out);
    return p.n_chunks > 1 ? (size_t)p.n_chunks * N_in * N_out * sizeof(float) : 256;
  }
  const DwPlan p = plan_dw_interleaved(T, B, N_in, N_out);
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
  Carve c(nullptr);
  if (N_out <= kNarrowOut) {  // padded dense G and delta
    c.take<float>((size_t)T * B * narrow_ld(N_out));
    c.take<float>((size_t)T * B * narrow_ld(N_out));
    return c.off;
  }
  const WalkPlan wp = plan_walk(T);
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
// Padded dense G of a narrow layer (N_out <= kNarrowOut), zeros included: [T*B][narrow_ld].
void enqueue_narrow_g(int TB, int N_out, const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                      const float* eps_out, int64_t out_cap, float* Gd, hipStream_t s) {
  const unsigned row_blocks = (unsigned)(((int64_t)TB * kWave + 255) / 256);
  hipLaunchKernelGGL(narrow_scatter_g, dim3(row_blocks), dim3(256), 0, s, TB, N_out, narrow_ld(N_out), out_row_ptr,
                     out_col_idx, out_g, eps_out, out_cap, Gd);
}

// dW of one layer. For a narrow layer the dense G goes to the front of the workspace; g_ready
// says it is there already (written by enqueue_narrow_g on this stream).
// The parts of a dW call: the layout depends only on the output CSR's structure (row pointers,
// columns); the rest needs eps too. kAll runs both.
enum DwPhase { kDwAll, kDwLayout, kDwRest };

void enqueue_dw(const float* trace_in, int T, int B, int N_in, int N_out, const int32_t* out_row_ptr,
                const int32_t* out_col_idx, const float* out_g, const float* eps_out, int64_t out_cap, float* dW,
                void* workspace, hipStream_t s, bool g_ready = false, DwPhase phase = kDwAll) {
  const bool layout = phase != kDwRest, rest = phase != kDwLayout;
  if (out_cap == 0) {  // no active output entry: dW = 0 and no entry array is read
    if (rest) fill_zero_async(dW, (size_t)N_in * N_out, s);
    return;
  }
  if (N_out <= kNarrowOut) {
    const int TB = T * B;
    const NarrowDwPlan q = plan_narrow_dw(T, B, N_in);
    Carve ws(workspace);
    float* Gd = ws.take<float>((size_t)TB * narrow_ld(N_out));
    uint64_t* busy = ws.take<uint64_t>(((size_t)TB + kWave - 1) / kWave);
    float* part = q.n_chunks > 1 ? ws.take<float>((size_t)q.n_chunks * N_in * N_out) : dW;
    if (layout)
      hipLaunchKernelGGL(narrow_busy_rows, dim3((unsigned)((TB + 255) / 256)), dim3(256), 0, s, TB, out_row_ptr,
                         out_cap, busy);
    if (!rest) return;
    if (!g_ready) enqueue_narrow_g(TB, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, Gd, s);
    // columns in blocks of 8 (N_out <= 8) or 16 (grid y: one or two blocks)
    const int ld = narrow_ld(N_out);
    const unsigned blocks = (unsigned)(((int64_t)q.n_chunks * q.n_iw * kWave + 255) / 256);
    if (ld == 8)
      hipLaunchKernelGGL(narrow_dw<8>, dim3(blocks), dim3(256), 0, s, trace_in, TB, N_in, N_out, busy, Gd, ld,
                         q.rows_per_chunk, q.n_iw, part);
    else
      hipLaunchKernelGGL(narrow_dw<16>, dim3(blocks, (unsigned)(ld / 16)), dim3(256), 0, s, trace_in, TB, N_in, N_out,
                         busy, Gd, ld, q.rows_per_chunk, q.n_iw, part);
    if (q.n_chunks > 1) {
      const int64_t n = (int64_t)N_in * N_out;
      hipLaunchKernelGGL(narrow_reduce, dim3((unsigned)((n + kWave - 1) / kWave)), dim3(kReduceWaves * kWave), 0, s,
                         part, q.n_chunks, n, dW);
    }
    return;
  }
  if (mdw_eligible(T, B, N_in, N_out, out_cap)) {  // matrix-core accumulation over windows sorted by column quad
    if (layout) mdw_enqueue_layout(T, B, N_in, N_out, out_row_ptr, out_col_idx, out_cap, workspace, s);
    if (rest) mdw_enqueue_rest(trace_in, T, B, N_in, N_out, out_g, eps_out, out_cap, dW, workspace, s);
    return;
  }
  if (dw_rows_eligible(N_in, N_out)) {  // straight from the CSR: no layout pass
    if (!rest) return;
    const DwPlan p = plan_dw_rows(T, B, N_in, N_out);
    float* part = p.n_chunks > 1 ? static_cast<float*>(workspace) : dW;
    const dim3 grid((unsigned)(p.n_itiles * p.n_chunks));
    if (out_g) {
      ensure_dynamic_lds((const void*)dw_rows_kernel<true>, (int)p.lds);
      hipLaunchKernelGGL(dw_rows_kernel<true>, grid, dim3(kDwThreads), p.lds, s, trace_in, T * B, N_in, N_out,
                         out_row_ptr, out_col_idx, out_g, eps_out, out_cap, part, p.n_chunks, p.n_itiles);
    } else {
      ensure_dynamic_lds((const void*)dw_rows_kernel<false>, (int)p.lds);
      hipLaunchKernelGGL(dw_rows_kernel<false>, grid, dim3(kDwThreads), p.lds, s, trace_in, T * B, N_in, N_out,
                         out_row_ptr, out_col_idx, out_g, eps_out, out_cap, part, p.n_chunks, p.n_itiles);
    }
    if (p.n_chunks > 1) {
      const size_t n = (size_t)N_in * N_out;
      const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
      hipLaunchKernelGGL(reduce_chunks, dim3(blocks), dim3(256), 0, s, part, p.n_chunks, n, dW);
    }
    return;
  }
  const int TB = T * B;
  const DwPlan p = plan_dw_interleaved(T, B, N_in, N_out);
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
  if (layout) {
    hipLaunchKernelGGL(slab_count, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr, out_col_idx,
                       out_cap, scnt);
    launch_exclusive_scan(scnt, nsp, sp, nullptr, stmp, s);
  }
  if (!rest) return;
  if (out_g)
    hipLaunchKernelGGL(slab_fill<true>, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr,
                       out_col_idx, out_g, eps_out, out_cap, sp, nrec, rec);
  else
    hipLaunchKernelGGL(slab_fill<false>, rgrid, rblock, 0, s, TB, N_out, p.n_slabs, p.slab, R, out_row_ptr,
                       out_col_idx, out_g, eps_out, out_cap, sp, nrec, rec);
  const dim3 dgrid((unsigned)(p.n_itiles * p.n_slabs * p.n_chunks));
  ensure_dynamic_lds((const void*)dw_slab_kernel, (int)p.lds);
  hipLaunchKernelGGL(dw_slab_kernel, dgrid, dim3(kDwThreads), p.lds, s, trace_in, TB, N_in, N_out, sp, rec, nrec,
                     part, p.n_chunks, p.n_itiles, p.n_slabs, p.slab);
  if (p.n_chunks > 1) {
    const size_t n = (size_t)N_in * N_out;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(reduce_chunks, dim3(blocks), dim3(256), 0, s, part, p.n_chunks, n, dW);
  }
}

// Chunks of the trace-recompute dW: 128 samples x tlen steps (tlen a multiple of K), about as
// many as plan_dw's row chunks.
struct SpikesPlan {
  DwPlan base;
  int tlen, n_tblk, n_bblk, n_chunks;
};

SpikesPlan plan_dw_spikes(int T, int B, int N_in, int N_out, int K) {
  SpikesPlan q{};
  q.base = plan_dw(T, B, N_in, N_out);
  q.n_bblk = (B + kSamplesPerChunk - 1) / kSamplesPerChunk;
  const int want = std::max(1, q.base.n_chunks / q.n_bblk);  // chunks along time
  int tlen = (T + want - 1) / want;
  tlen = ((tlen + K - 1) / K) * K;
  q.tlen = tlen;
  q.n_tblk = (T + tlen - 1) / tlen;
  q.n_chunks = q.n_tblk * q.n_bblk;
  return q;
}

size_t dw_spikes_workspace(int T, int B, int N_in, int N_out, int64_t out_cap, int K) {
  const SpikesPlan q = plan_dw_spikes(T, B, N_in, N_out, K);
  const int nsp = q.base.n_slabs * T * B;
  Carve c(nullptr);
  if (q.n_chunks > 1) c.take<float>((size_t)q.n_chunks * N_in * N_out);
  c.take<int32_t>((size_t)nsp + 1);
  c.take<int32_t>((size_t)nsp);
  c.take<int32_t>(scan_temp_elems(nsp));
  c.take<SlabRec>((size_t)std::max<int64_t>(out_cap, 1));
  return c.off;
}

void enqueue_dw_spikes(const uint8_t* s_in, const float* ck, int K, float alpha, int T, int B, int N_in, int N_out,
                       const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                       const float* eps_out, int64_t out_cap, float* dW, void* workspace, hipStream_t s) {
  if (out_cap == 0) {
    fill_zero_async(dW, (size_t)N_in * N_out, s);
    return;
  }
  const int TB = T * B;
  const SpikesPlan q = plan_dw_spikes(T, B, N_in, N_out, K);
  const DwPlan& p = q.base;
  Carve ws(workspace);
  float* part = q.n_chunks > 1 ? ws.take<float>((size_t)q.n_chunks * N_in * N_out) : dW;
  const int nsp = p.n_slabs * TB;
  int32_t* sp = ws.take<int32_t>((size_t)nsp + 1);
  int32_t* scnt = ws.take<int32_t>((size_t)nsp);
  int32_t* stmp = ws.take<int32_t>(scan_temp_elems(nsp));
  SlabRec* rec = ws.take<SlabRec>((size_t)std::max<int64_t>(out_cap, 1));
  const int R = std::max(1, std::min(8, kWave / p.n_slabs));
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
  const dim3 dgrid((unsigned)(p.n_itiles * p.n_slabs * q.n_chunks));
  ensure_dynamic_lds((const void*)dw_slab_spikes_kernel, (int)p.lds);
  hipLaunchKernelGGL(dw_slab_spikes_kernel, dgrid, dim3(kDwThreads), p.lds, s, s_in, ck, K, alpha, T, B, N_in, N_out,
                     sp, rec, nrec, part, q.tlen, q.n_bblk, p.n_itiles, p.n_slabs, p.slab);
  if (q.n_chunks > 1) {
    const size_t n = (size_t)N_in * N_out;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(reduce_chunks, dim3(blocks), dim3(256), 0, s, part, q.n_chunks, n, dW);
  }
}

// Spike gradient of one layer: chunk sums, carries, the walk. share_cu keeps the walk to two
// blocks per CU so that a kernel running beside it (dW) finds room. Arguments already validated.
void enqueue_grad_in(const float* W, int T, int B, int N_in, int N_out, float alpha, const int32_t* out_row_ptr,
                     const int32_t* out_col_idx, const float* out_g, const float* eps_out, int64_t out_cap,
                     const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap, float* eps_in,
                     bool share_cu, void* workspace, hipStream_t s, const float* g_dense = nullptr) {
  if (in_cap == 0) return;
  if (out_cap == 0) {  // no active output entry: delta = 0 everywhere
    fill_zero_async(eps_in, (size_t)in_cap, s);
    return;
  }
  if (N_out <= kNarrowOut) {
    const int ld = narrow_ld(N_out);
    Carve ws(workspace);
    const size_t n = (size_t)T * B * ld;
    float* Gd = ws.take<float>(n);
    float* D = ws.take<float>(n);
    const int TB = T * B;
    if (g_dense)
      Gd = const_cast<float*>(g_dense);
    else
      enqueue_narrow_g(TB, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, Gd, s);
    const int64_t BL = (int64_t)B * ld;
    hipLaunchKernelGGL(narrow_delta, dim3((unsigned)((BL + 255) / 256)), dim3(256), 0, s, T, BL, alpha, Gd, D);
    const unsigned row_blocks = (unsigned)(((int64_t)TB * kWave + 255) / 256);
#define SNN_NGIN(NJ_)                                                                                        \
  hipLaunchKernelGGL(narrow_gin<NJ_>, dim3(row_blocks), dim3(256), 0, s, TB, N_in, N_out, W, D, in_row_ptr, \
                     in_col_idx, in_cap, eps_in)
    if (ld == 8) SNN_NGIN(8);
    else if (ld == 16) SNN_NGIN(16);
    else SNN_NGIN(32);
#undef SNN_NGIN
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
  const dim3 walk_grid(share_cu ? std::min<unsigned>(wgrid.x, 2u * (unsigned)cu_count()) : wgrid.x);
  if (nj > 4 && N_out % 4 == 0) {
#define SNN_WALK4(NJ_)                                                                                        \
  launch_walk_x4<NJ_>(walk_grid, s, W, T, B, N_in, N_out, alpha, wp.P, wp.C, out_row_ptr, out_col_idx, out_g, \
                      eps_out, out_cap, in_row_ptr, in_col_idx, in_cap, Lbuf, eps_in)
    if (nj <= 8) SNN_WALK4(8);
    else if (nj <= 16) SNN_WALK4(16);
    else if (nj <= 32) SNN_WALK4(32);
    else SNN_WALK4(64);
#undef SNN_WALK4
    return;
  }
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

extern "C" snn_status snn_sparse_dw_layout(int T, int B, int N_in, int N_out, const int32_t* out_row_ptr,
                                           const int32_t* out_col_idx, int64_t out_cap, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  if (!dims_ok(T, B, N_in, N_out) || !out_row_ptr || out_cap < 0 || (out_cap > 0 && !out_col_idx))
    return SNN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < dw_workspace(T, B, N_in, N_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;
  enqueue_dw(nullptr, T, B, N_in, N_out, out_row_ptr, out_col_idx, nullptr, nullptr, out_cap, nullptr, workspace,
             static_cast<hipStream_t>(stream), false, kDwLayout);
  return launch_status();
}

extern "C" snn_status snn_sparse_dw_prepared(const float* trace_in, int T, int B, int N_in, int N_out,
                                             const int32_t* out_row_ptr, const int32_t* out_col_idx,
                                             const float* out_g, const float* eps_out, int64_t out_cap, float* dW,
                                             void* workspace, size_t workspace_bytes, void* stream) {
  if (!trace_in || !dW || !dims_ok(T, B, N_in, N_out)) return SNN_ERR_INVALID_ARG;
  if (!out_csr_ok(out_row_ptr, out_col_idx, eps_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < dw_workspace(T, B, N_in, N_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;
  enqueue_dw(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, workspace,
             static_cast<hipStream_t>(stream), false, kDwRest);
  return launch_status();
}

extern "C" int64_t snn_trace_checkpoint_count(int T, int K) {
  if (bad_dim(T) || bad_dim(K)) return 0;
  return (T + K - 1) / K;
}

extern "C" snn_status snn_trace_checkpoints(const uint8_t* s_in, int T, int B, int N_in, float alpha, int K, float* ck,
                                            void* stream) {
  if (!s_in || !ck || bad_dim(T) || bad_dim(B) || bad_dim(N_in) || bad_dim(K) || too_big(T, B, N_in))
    return SNN_ERR_INVALID_ARG;
  if (bad_alpha(alpha)) return SNN_ERR_INVALID_ARG;
  const int64_t n = (int64_t)B * N_in;
  hipLaunchKernelGGL(trace_checkpoints_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), s_in, T, B, N_in, alpha, K, ck);
  return launch_status();
}

extern "C" size_t snn_sparse_dw_spikes_workspace(int T, int B, int N_in, int N_out, int64_t out_cap, int K) {
  if (!dims_ok(T, B, N_in, N_out) || out_cap < 0 || bad_dim(K)) return 0;
  return dw_spikes_workspace(T, B, N_in, N_out, out_cap, K);
}

extern "C" snn_status snn_sparse_dw_spikes(const uint8_t* s_in, const float* ck, int K, float alpha, int T, int B,
                                           int N_in, int N_out, const int32_t* out_row_ptr,
                                           const int32_t* out_col_idx, const float* out_g, const float* eps_out,
                                           int64_t out_cap, float* dW, void* workspace, size_t workspace_bytes,
                                           void* stream) {
  if (!s_in || !ck || !dW || !dims_ok(T, B, N_in, N_out) || bad_dim(K) || bad_alpha(alpha))
    return SNN_ERR_INVALID_ARG;
  if (!out_csr_ok(out_row_ptr, out_col_idx, eps_out, out_cap)) return SNN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < dw_spikes_workspace(T, B, N_in, N_out, out_cap, K)) return SNN_ERR_INVALID_ARG;
  if (N_out > 4096) return SNN_ERR_UNSUPPORTED;
  enqueue_dw_spikes(s_in, ck, K, alpha, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW,
                    workspace, static_cast<hipStream_t>(stream));
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

namespace {
// The fork and join events of snn_sparse_backward's auxiliary stream: two per device and host
// thread, created on first use and kept for the life of the thread, so that a call creates and
// destroys nothing. A stream wait takes the event's state when it is enqueued, so reusing the
// pair call after call on one thread is safe.
bool fork_join_events(hipEvent_t* in, hipEvent_t* out) {
  constexpr int kMaxDevices = 64;
  thread_local hipEvent_t ev[kMaxDevices][2] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
  for (int k = 0; k < 2; ++k)
    if (!ev[dev][k] && hipEventCreateWithFlags(&ev[dev][k], hipEventDisableTiming) != hipSuccess) {
      ev[dev][k] = nullptr;
      return false;
    }
  *in = ev[dev][0];
  *out = ev[dev][1];
  return true;
}
}  // namespace

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
  // A narrow layer's dense G is written once, at the front of the dW workspace, before the fork.
  const bool narrow_g = N_out <= kNarrowOut && out_cap > 0;
  if (narrow_g)
    enqueue_narrow_g(T * B, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, reinterpret_cast<float*>(dw_ws),
                     s);
  // The spike gradient (a gather of W rows) and dW (matrix cores on LDS tiles) lean on different
  // parts of a CU; with an auxiliary stream they run side by side. aux waits for what is already
  // on s, and s waits for aux before anything enqueued after this call.
  hipStream_t sa = s;
  hipEvent_t ev_in = nullptr, ev_out = nullptr;
  if (do_gin && aux_stream && aux_stream != stream && fork_join_events(&ev_in, &ev_out)) {
    if (hipEventRecord(ev_in, s) != hipSuccess ||
        hipStreamWaitEvent(static_cast<hipStream_t>(aux_stream), ev_in, 0) != hipSuccess)
      return SNN_ERR_HIP;  // nothing enqueued yet
    sa = static_cast<hipStream_t>(aux_stream);
  }
  if (do_gin) {
    // beside a dW that takes longer than the walk, the walk leaves room for a dW block on every
    // CU (per product, a dW entry costs about 1.5 times a walk entry)
    const bool dw_longer = 3.0 * (double)out_cap * N_in >= 2.0 * (double)in_cap * N_out;
    enqueue_grad_in(W, T, B, N_in, N_out, alpha, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, in_row_ptr,
                    in_col_idx, in_cap, eps_in, sa != s && dw_longer, gin_ws, sa,
                    narrow_g ? reinterpret_cast<const float*>(dw_ws) : nullptr);
  }
  enqueue_dw(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, dw_ws, s, narrow_g);
  if (sa != s && (hipEventRecord(ev_out, sa) != hipSuccess || hipStreamWaitEvent(s, ev_out, 0) != hipSuccess))
    return SNN_ERR_HIP;  // the join failed: later work on stream is not ordered after eps_in
  return launch_status();
}
