// Sparse weight gradient on the matrix cores (sparse form of Eq. (w_grad), Sec. 2.2):
//   dW[i, j] = sum over the active output entries (t, b, j) of G[t,b,j] * trace[t,b,i],
//   G = eps * g (Definition 2).
//
// Layout (structure only, runs as soon as the active set is known): rows r = t*B + b are cut into
// windows of kMRW rows, and each window's entries are sorted by column quad, in CSR order (row, then
// column) inside a quad. The sorted copy occupies the window's own CSR range, so the workspace is
// bounded by the CSR capacity. qoff[w][q] is where quad q of window w starts. Quads are formed after a
// permutation of the columns that balances their activity: the columns are ranked by their number of
// active entries over the whole batch and dealt to the quads in snake order (ranks 0..Q-1 to quads
// 0..Q-1, ranks Q..2Q-1 to quads Q-1..0, ...), so the sixteen quads of a wavefront, which advance in
// lockstep, carry similar numbers of entries even when a few neurons are far more active than most.
//
// Accumulation: v_mfma_f32_4x4x1f32 computes sixteen independent 4x4 outer products per instruction.
// A wavefront owns 64 inputs x 64 columns; block b of its MFMA (lanes 4b..4b+3) owns quad b of the
// wavefront's columns and, in each group of sixteen instructions, takes the next entry of that quad:
// its B operand is G at the entry's column (zero at the quad's other three columns), its A operand
// the entry's trace row, four inputs per lane. The sixteen accumulator tiles (one per four inputs)
// are fixed registers, so an entry's column never becomes a register index and no LDS atomics are
// needed. The trace rows of a window (64 inputs of the block's input tile) and the window's sorted
// entries are staged in LDS by direct global-to-LDS loads, double buffered: the next window's loads
// are in flight while the current window is accumulated. A window whose entries do not fit the LDS
// record area is processed in several rounds of whole quads.
//
// Blocks: (input tile of 64 inputs) x (chunk of windows: chunk c of n takes windows c, c + n, ...,
// so every chunk spans the whole time axis and the chunks end together wherever the activity lies
// in time; contiguous runs of windows made stress's dW calls 2-4% slower); each block writes a
// partial dW for its chunk with columns in slot order (a wavefront's 64 slots are contiguous, so the stores coalesce);
// mdw_reduce sums the partials in a fixed order in float64 and puts each column in its place, so
// dW is bitwise reproducible.
#include "common.h"
#include <climits>

namespace snn {
namespace {

constexpr int kMRW = 128;                       // rows per window
constexpr int kMStride = 320;                   // bytes per staged trace row: 64 inputs + 16 bytes (bank spread)
constexpr int kMQ = 256;                        // column quads per block (1024 columns)
constexpr int kMQLd = 260;                      // ints per qoff row (16-byte aligned rows)
constexpr int kMTr = kMRW * kMStride;           // 40960: trace tile
constexpr int kMRecB = 36 * 1024;               // record area (whole 1 KB pieces of direct loads)
constexpr int kMRC = kMRecB / 8 - 2;            // records per round (room for an odd start and a pair tail)
constexpr int kMQB = 2048;                      // qoff area (65 pieces of 16 bytes, whole 1 KB loads)
constexpr int kMBuf = kMTr + kMRecB + kMQB;     // one staging buffer
constexpr int kMThreads = 1024;
constexpr int kMWaves = kMThreads / kWave;      // 16 wavefronts x 64 columns = 1024 columns
constexpr int kMTile = 64;                      // inputs per block
static_assert(kMQLd * 4 % 16 == 0 && (kMQ + 1) <= kMQLd, "qoff rows are whole 16-byte pieces");
static_assert((kMQLd * 4 / 16) <= kMQB / 16 && kMQB % 1024 == 0, "qoff area holds a row");
static_assert(kMTr % 1024 == 0 && kMRecB % 1024 == 0, "direct loads write whole 1 KB pieces");
static_assert(2 * kMBuf <= 160 * 1024, "two staging buffers in LDS");
static_assert(kMRC >= 4 * kMRW, "a quad's entries of one window fit one round");

constexpr int kLayWaves = 4;
constexpr int kLayRows = kMRW / kLayWaves;

typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int clampi(int v, int64_t cap) { return (int)(v < 0 ? 0 : (v > cap ? cap : v)); }

// One 16-byte direct global-to-LDS load per lane into 64 consecutive 16-byte LDS slots starting at
// the wave-uniform LDS byte address lds. Issued through inline asm so that the compiler does not
// order every later LDS read behind it; callers wait with s_waitcnt vmcnt(0) before the data is read.
__device__ __forceinline__ void mdw_dma16(const void* g, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(g) : "memory", "m0");
}

__device__ __forceinline__ void mdw_wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, kWave));
  return v;
}

// Active entries per column over the whole CSR (entries [0, min(nnz, cap)) with a valid column):
// per-block LDS histograms added into cnt (zeroed beforehand by mdw_zero).
__global__ void mdw_zero(int32_t* __restrict__ p, int n) {
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) p[k] = 0;
}

__global__ __launch_bounds__(256) void mdw_colcount(int TB, int N_out, const int32_t* __restrict__ row_ptr,
                                                    const int32_t* __restrict__ col_idx, int64_t cap,
                                                    int32_t* __restrict__ cnt) {
  __shared__ int h[kMQ * 4];
  for (int k = threadIdx.x; k < N_out; k += blockDim.x) h[k] = 0;
  __syncthreads();
  const int n = clampi(row_ptr[TB], cap);
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) {
    const int c = col_idx[e];
    if ((unsigned)c < (unsigned)N_out) atomicAdd(&h[c], 1);
  }
  __syncthreads();
  for (int k = threadIdx.x; k < N_out; k += blockDim.x)
    if (h[k]) atomicAdd(&cnt[k], h[k]);
}

// Column c's rank (descending count, ties by index) gives its slot v in the quad layout (snake
// dealing over nq = ceil(N_out / 4) quads): perm[c] = v, inv[v] = c, and inv[v] = -1 for the slots
// of ranks N_out .. 4 nq - 1 (no column). Each block ranks 64 columns; its four wavefronts split
// the comparisons and add their partial ranks in LDS. (Small blocks: this runs on a side stream
// beside other kernels and must find room on a busy compute unit.)
constexpr int kPermWaves = 4;
constexpr int kPermCmp = kMQ * 4 / kPermWaves;  // comparisons per wavefront
__global__ __launch_bounds__(kPermWaves * kWave) void mdw_perm(int N_out, const int32_t* __restrict__ cnt,
                                                               int32_t* __restrict__ perm, int32_t* __restrict__ inv) {
  __shared__ __attribute__((aligned(16))) int cs[kMQ * 4];
  __shared__ int part[kPermWaves][kWave];
  const int t = threadIdx.x;
  const int nq = (N_out + 3) / 4;
  for (int k = t; k < kMQ * 4; k += blockDim.x) cs[k] = k < N_out ? cnt[k] : INT_MIN;
  __syncthreads();
  const int l = t & (kWave - 1), w = t / kWave;
  const int c = blockIdx.x * kWave + l;
  const int mine = c < N_out ? cs[c] : 0;
  int rank = 0;
  const int k0 = w * kPermCmp;  // this wavefront's comparisons (entries past N_out hold INT_MIN)
#pragma unroll 4
  for (int k = k0; k < k0 + kPermCmp; k += 4) {
    const int4 o = *reinterpret_cast<const int4*>(cs + k);
    rank += (o.x > mine) || (o.x == mine && k < c);
    rank += (o.y > mine) || (o.y == mine && k + 1 < c);
    rank += (o.z > mine) || (o.z == mine && k + 2 < c);
    rank += (o.w > mine) || (o.w == mine && k + 3 < c);
  }
  part[w][l] = rank;
  __syncthreads();
  auto slot_of = [nq](int r) {
    const int round = r / nq, idx = r - round * nq;
    return 4 * ((round & 1) ? nq - 1 - idx : idx) + round;
  };
  if (w == 0 && c < N_out) {
    int r = 0;
#pragma unroll
    for (int k = 0; k < kPermWaves; ++k) r += part[k][l];
    const int v = slot_of(r);
    perm[c] = v;
    inv[v] = c;
  }
  if (blockIdx.x == 0 && N_out + t < 4 * nq) inv[slot_of(N_out + t)] = -1;  // at most three
}

// Layout: one block per window. The window's entries (its CSR range) are split into four contiguous
// parts, one per wavefront. Pass 1 counts each part's entries per quad; pass 2 gives each entry its
// slot: the quad's start, the quad's entries in earlier parts, this part's running count and the
// entry's place among the same quad's entries of its 64-entry piece (a match mask from one ballot
// per bit of the quad). CSR order is kept inside a quad. Writes rec[slot].x = row offset in the
// trace tile | (column slot % 4) << 20, src[slot] = entry index, and the window's qoff row
// (absolute entry positions; qoff[256] = end of the window's valid entries).
__global__ __launch_bounds__(kLayWaves * kWave) void mdw_layout(int TB, int N_out, const int32_t* __restrict__ row_ptr,
                                                                const int32_t* __restrict__ col_idx, int64_t cap,
                                                                const int32_t* __restrict__ perm,
                                                                int32_t* __restrict__ qoff, int2* __restrict__ rec,
                                                                int32_t* __restrict__ src) {
  __shared__ int cnt[kLayWaves][kMQ];
  __shared__ int rp[kMRW + 1];
  __shared__ int pm[kMQ * 4];
  const int w = threadIdx.x / kWave;
  const int l = lane_id();
  const int win = blockIdx.x;
  const int r0 = win * kMRW;
  const int nr = min(kMRW, TB - r0);
  for (int k = threadIdx.x; k <= nr; k += blockDim.x) rp[k] = clampi(row_ptr[r0 + k], cap);
  for (int k = threadIdx.x; k < kLayWaves * kMQ; k += blockDim.x) (&cnt[0][0])[k] = 0;
  for (int k = threadIdx.x; k < N_out; k += blockDim.x) pm[k] = perm[k];
  __syncthreads();
  const int e_a = rp[0];
  const int len = max(rp[nr] - e_a, 0);
  const int pa = e_a + (int)((int64_t)len * w / kLayWaves);
  const int pb = e_a + (int)((int64_t)len * (w + 1) / kLayWaves);
  for (int e = pa + l; e < pb; e += kWave) {
    const int c = col_idx[e];
    if ((unsigned)c < (unsigned)N_out) atomicAdd(&cnt[w][pm[c] >> 2], 1);  // counts only: order does not matter
  }
  __syncthreads();
  if (w == 0) {  // exclusive scan over quads (lane: quads 4l..4l+3), then the per-part starts
    int tot[4], s = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      tot[k] = 0;
#pragma unroll
      for (int q = 0; q < kLayWaves; ++q) tot[k] += cnt[q][4 * l + k];
      s += tot[k];
    }
    int run = e_a + wave_incl_scan(s) - s;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int quad = 4 * l + k;
      qoff[(size_t)win * kMQLd + quad] = run;
      int b = run;
#pragma unroll
      for (int q = 0; q < kLayWaves; ++q) {
        const int c = cnt[q][quad];
        cnt[q][quad] = b;
        b += c;
      }
      run += tot[k];
    }
    if (l == kWave - 1) qoff[(size_t)win * kMQLd + kMQ] = run;
  }
  __syncthreads();
  const uint64_t below = (1ull << l) - 1ull;
  for (int e0 = pa; e0 < pb; e0 += kWave) {
    const int e = e0 + l;
    const int c = e < pb ? col_idx[e] : -1;
    const bool valid = (unsigned)c < (unsigned)N_out;
    const int v = valid ? pm[c] : 0;           // the column's slot in the quad layout
    const int key = valid ? (v >> 2) : 511;    // quads < 256; 511 marks lanes without an entry
    uint64_t match = ~0ull;
#pragma unroll
    for (int bit = 0; bit < 9; ++bit) {
      const uint64_t bal = __ballot((key >> bit) & 1);
      match &= ((key >> bit) & 1) ? bal : ~bal;
    }
    const int before = __popcll(match & below);
    const int after = __popcll(match & ~below & ~(1ull << l));
    // the entry's row: last r with rp[r] <= e (rows of the window only)
    int lo = 0, hi = nr - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (rp[mid] <= e) lo = mid; else hi = mid - 1;
    }
    const int base = valid ? cnt[w][key] : 0;
    const int slot = base + before;
    if (valid && slot < cap) {  // a malformed CSR cannot write past the arrays
      rec[slot].x = (lo * kMStride) | ((v & 3) << 20);
      src[slot] = e;
    }
    __builtin_amdgcn_wave_barrier();
    if (valid && after == 0) cnt[w][key] = slot + 1;
  }
}

// G = eps * g into the sorted copy (the part that needs eps).
__global__ void mdw_gate(const int32_t* __restrict__ qoff, int64_t cap, const int32_t* __restrict__ src,
                         const float* __restrict__ g, const float* __restrict__ eps, int2* __restrict__ rec) {
  const int win = blockIdx.x;
  const int a = clampi(qoff[(size_t)win * kMQLd], cap);
  const int z = clampi(qoff[(size_t)win * kMQLd + kMQ], cap);
  // kAhead entries per thread at a time: their indices, then their eps and g, are all requested
  // before any is used (one dependent round trip per kAhead entries instead of per entry)
  constexpr int kAhead = 8;
  const int step = (int)blockDim.x;
  for (int d0 = a + threadIdx.x; d0 < z; d0 += kAhead * step) {
    int e[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      const int d = d0 + u * step;
      e[u] = d < z ? clampi(src[d], cap - 1) : 0;
    }
    float v[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) v[u] = g ? eps[e[u]] * g[e[u]] : eps[e[u]];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      const int d = d0 + u * step;
      if (d < z) rec[d].y = __float_as_int(v[u]);
    }
  }
}

// The accumulation (see the file comment). Block -> (input tile it, chunk ch); when the grid allows,
// the blocks of one chunk run on one XCD (the dispatcher deals blocks to the 8 XCDs in turn), so the
// chunk's sorted entries come from HBM once and are then shared through that XCD's L2.
__global__ __launch_bounds__(kMThreads) void mdw_kernel(const float* __restrict__ trace, int TB, int N_in, int N_out,
                                                        const int32_t* __restrict__ qoff, const int2* __restrict__ rec,
                                                        const int32_t* __restrict__ inv, int64_t cap, int n_win,
                                                        int n_itiles, float* __restrict__ part, bool chunked) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int it, ch;
  if ((gridDim.x & 7) == 0 && ((gridDim.x >> 3) % n_itiles) == 0) {
    const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
    it = j % n_itiles;
    ch = (j / n_itiles) * 8 + x;
  } else {
    it = blockIdx.x % n_itiles;
    ch = blockIdx.x / n_itiles;
  }
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int l = lane_id();
  const int t = l & 3;
  const int quad = 16 * w + (l >> 2);  // this lane group's column quad
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  const int i0 = it * kMTile;
  f4v C[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) C[q] = f4v{0.f, 0.f, 0.f, 0.f};
  // chunk ch takes windows ch, ch + nch, ch + 2 nch, ...: every chunk spans the whole time axis
  const int nch = (int)gridDim.x / n_itiles;
  auto win_of = [&](int k) { return ch + k * nch; };

  // Direct loads of window win into buffer bi: its trace rows (input tile it; lanes past the row's
  // 64 inputs fill the padding), its first round of sorted entries and its qoff row. Every source
  // address is clamped into its array.
  // e_lo / e_hi: the window's entry range (read before the loads are issued: a later global read
  // would wait for them too, vmcnt being in order).
  auto stage = [&](int bi, int win, int e_lo, int e_hi) {
    const unsigned base = lds0 + (unsigned)(bi * kMBuf);
    if (e_hi == e_lo) return;
    const int r0 = win * kMRW;
    const int nrows = min(kMRW, TB - r0);
    const int pieces = nrows * (kMStride / 16);
    for (int k = w; k * kWave < pieces; k += kMWaves) {
      const int p = k * kWave + l;
      const int row = p / (kMStride / 16), cc = p % (kMStride / 16);
      const int in = i0 + cc * 4;
      const bool ok = p < pieces && cc < kMTile / 4 && in < N_in;
      const float* s = trace + (ok ? (size_t)(r0 + row) * N_in + in : 0);
      mdw_dma16(s, __builtin_amdgcn_readfirstlane(base + k * 1024));
    }
    const int ea = e_lo & ~1;
    const int eb = min(e_hi, e_lo + kMRC);
    const int rpieces = (eb - ea + 1) >> 1;
    const int last = (int)((cap + 2) >> 1);  // last whole 16-byte piece of the record array (cap + 4 records)
    for (int k = w; k * kWave < rpieces; k += kMWaves) {
      const int p = min(k * kWave + l, rpieces - 1);
      const int pc = min((ea >> 1) + p, last);
      mdw_dma16(reinterpret_cast<const int4*>(rec) + pc, __builtin_amdgcn_readfirstlane(base + kMTr + k * 1024));
    }
    if (w == 0) {  // the qoff row: 65 pieces, two loads (the second one's lanes all take piece 64)
      const int4* qrow = reinterpret_cast<const int4*>(qoff + (size_t)win * kMQLd);
      mdw_dma16(qrow + l, __builtin_amdgcn_readfirstlane(base + kMTr + kMRecB));
      mdw_dma16(qrow + kMQLd * 4 / 16 - 1, __builtin_amdgcn_readfirstlane(base + kMTr + kMRecB + 1024));
    }
  };

  // Entry ranges of the chunk's windows, 64 at a time: lane l holds the chunk's window 64 g + l. A
  // group is loaded right after a barrier, before any staging load is in flight.
  int rng_lo = 0, rng_hi = 0;
  auto range_of = [&](int k, int& lo, int& hi) {
    if ((k & (kWave - 1)) == 0) {
      const int wv = win_of(k + l);
      const int a = wv < n_win ? clampi(qoff[(size_t)wv * kMQLd], cap) : 0;
      rng_lo = a;
      rng_hi = wv < n_win ? max(a, clampi(qoff[(size_t)wv * kMQLd + kMQ], cap)) : 0;
    }
    lo = __builtin_amdgcn_readlane(rng_lo, k & (kWave - 1));
    hi = __builtin_amdgcn_readlane(rng_hi, k & (kWave - 1));
  };
  int cur_lo = 0, cur_hi = 0;
  if (win_of(0) < n_win) {
    range_of(0, cur_lo, cur_hi);
    stage(0, win_of(0), cur_lo, cur_hi);
  }
  for (int k = 0; win_of(k) < n_win; ++k) {
    const int bi = k & 1;
    char* buf = smem + bi * kMBuf;
    mdw_wait_dma();
    __syncthreads();
    int nxt_lo = 0, nxt_hi = 0;
    if (win_of(k + 1) < n_win) {
      range_of(k + 1, nxt_lo, nxt_hi);
      stage(bi ^ 1, win_of(k + 1), nxt_lo, nxt_hi);
    }
    const int e_lo = cur_lo, e_hi = cur_hi;
    cur_lo = nxt_lo;
    cur_hi = nxt_hi;
    if (e_hi > e_lo) {
      const int* qs = reinterpret_cast<const int*>(buf + kMTr + kMRecB);
      const char* lb = buf + 16 * t;
      const int2* rl = reinterpret_cast<const int2*>(buf + kMTr);
      int base = e_lo, qa = 0;
      for (int round = 0; qa < kMQ; ++round) {
        // quads [qa, qb) whose entries fit the record area from base
        int qb = kMQ;
        if (e_hi - base > kMRC) {
          int lo = qa + 1, hi = kMQ;  // largest qb with qs[qb] - base <= kMRC (at least qa + 1)
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (clampi(qs[mid], cap) - base <= kMRC) lo = mid; else hi = mid - 1;
          }
          qb = lo;
        }
        const int ra = base & ~1;
        if (round > 0) {  // a dense window: this round's entries are loaded now
          __syncthreads();
          const int eb = min(e_hi, base + kMRC);
          const int rpieces = (eb - ra + 1) >> 1;
          const int last = (int)((cap + 2) >> 1);
          const unsigned rbase = lds0 + (unsigned)(bi * kMBuf + kMTr);
          for (int k = w; k * kWave < rpieces; k += kMWaves) {
            const int p = min(k * kWave + l, rpieces - 1);
            mdw_dma16(reinterpret_cast<const int4*>(rec) + min((ra >> 1) + p, last),
                      __builtin_amdgcn_readfirstlane(rbase + k * 1024));
          }
          mdw_wait_dma();
          __syncthreads();
        }
        const bool mine = quad >= qa && quad < qb;
        int lo = mine ? clampi(qs[quad], cap) : 0;
        int hi = mine ? clampi(qs[quad + 1], cap) : 0;
        lo = max(lo, base);
        hi = min(max(hi, lo), base + kMRC);
        const int len = mine ? hi - lo : 0;
        const int K = wave_max(len);
        const int off = lo - ra;
        for (int k = 0; k < K; ++k) {
          int2 rc = make_int2(0, 0);
          if (k < len) rc = rl[off + k];
          const char* p = lb + (rc.x & 0xFFFF);
          const float Bv = ((rc.x >> 20) & 3) == t ? __int_as_float(rc.y) : 0.0f;
          float4 av[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) av[q] = *reinterpret_cast<const float4*>(p + 64 * q);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            C[4 * q + 0] = __builtin_amdgcn_mfma_f32_4x4x1f32(av[q].x, Bv, C[4 * q + 0], 0, 0, 0);
            C[4 * q + 1] = __builtin_amdgcn_mfma_f32_4x4x1f32(av[q].y, Bv, C[4 * q + 1], 0, 0, 0);
            C[4 * q + 2] = __builtin_amdgcn_mfma_f32_4x4x1f32(av[q].z, Bv, C[4 * q + 2], 0, 0, 0);
            C[4 * q + 3] = __builtin_amdgcn_mfma_f32_4x4x1f32(av[q].w, Bv, C[4 * q + 3], 0, 0, 0);
          }
        }
        base = max(base, clampi(qs[qb], cap));
        qa = qb;
      }
    }
    __syncthreads();  // every wavefront is done with this buffer before it is staged again
  }
  // C[4q + u] register v, lane 4b + j: input i0 + 16q + 4v + u, column slot 64w + 4b + j (column inv[slot])
  const int slot = kWave * w + l;
  const int S = 4 * ((N_out + 3) / 4);  // column slots per row
  if (chunked) {  // partial of chunk ch, rows of S slots (mdw_reduce applies the column order)
    float* dst = part + (size_t)ch * N_in * S;
    if (slot < S) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int i = i0 + 16 * q + 4 * v + u;
            if (i < N_in) dst[(size_t)i * S + slot] = C[4 * q + u][v];
          }
    }
  } else {  // one chunk: straight into dW, column inv[slot]
    const int col = slot < S ? inv[slot] : -1;
    if (col >= 0 && col < N_out) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int i = i0 + 16 * q + 4 * v + u;
            if (i < N_in) part[(size_t)i * N_out + col] = C[4 * q + u][v];
          }
    }
  }
}

// dW = sum of the chunk partials in chunk order, float64 (deterministic); 256 outputs per block.
// Partials are rows of S column slots, read in slot order (coalesced); slot v goes to column
// inv[v] of dW (slots without a column hold -1 and are skipped).
__global__ __launch_bounds__(256) void mdw_reduce(const float* __restrict__ part, int n_chunks, int N_in, int N_out,
                                                  int S, const int32_t* __restrict__ inv, float* __restrict__ out) {
  const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = (int64_t)N_in * S;
  if (k >= n) return;
  const int64_t i = k / S;
  const int col = inv[k - i * S];
  if (col < 0 || col >= N_out) return;
  constexpr int kAhead = 8;  // partials loaded before any is added (the adds keep chunk order)
  double s = 0.0;
  int ch = 0;
  for (; ch + kAhead <= n_chunks; ch += kAhead) {
    float v[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) v[u] = part[(ch + u) * n + k];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) s += (double)v[u];
  }
  for (; ch < n_chunks; ++ch) s += (double)part[ch * n + k];
  out[i * N_out + col] = (float)s;
}

}  // namespace

// A block's sixteen wavefronts own 64 columns each; below 512 columns more than half of them would
// idle, and the slab kernels are as fast there (measured at 200, 300 and 400 columns). Above ~10%
// of the entries active (the capacity is the compaction's count) a window's entries need several
// record rounds and the lockstep quads cost more than the slab kernel's atomics (stress at 27%
// active: 67 against 45 ms); the dense chain is the faster one there anyway.
bool mdw_eligible(int T, int B, int N_in, int N_out, int64_t out_cap) {
  if (N_out < kMWaves * kWave / 2 || N_out > kMWaves * kWave || N_in % 4 != 0) return false;
  return (double)out_cap <= 0.1 * (double)T * (double)B * (double)N_out;
}

MdwPlan plan_mdw(int T, int B, int N_in, int N_out) {
  MdwPlan p{};
  (void)N_out;
  const int TB = T * B;
  p.n_win = (TB + kMRW - 1) / kMRW;
  p.n_itiles = (N_in + kMTile - 1) / kMTile;
  const int cus = cu_count();
  int nc = (cus + p.n_itiles - 1) / p.n_itiles;  // one block per CU (LDS), all CUs busy
  if (nc >= 8) nc = (nc + 7) / 8 * 8;             // whole XCD groups of chunks
  nc = std::max(1, std::min(nc, p.n_win));
  p.wpc = (p.n_win + nc - 1) / nc;
  p.n_chunks = (p.n_win + p.wpc - 1) / p.wpc;
  return p;
}

size_t mdw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap) {
  const MdwPlan p = plan_mdw(T, B, N_in, N_out);
  Carve c(nullptr);
  if (p.n_chunks > 1) c.take<float>((size_t)p.n_chunks * N_in * (4 * ((N_out + 3) / 4)));
  c.take<int32_t>((size_t)p.n_win * kMQLd);
  c.take<int2>((size_t)out_cap + 4);
  c.take<int32_t>((size_t)out_cap + 1);
  c.take<int32_t>((size_t)N_out);          // entries per column
  c.take<int32_t>((size_t)N_out);          // perm
  c.take<int32_t>((size_t)N_out + 4);      // inv
  return c.off;
}

namespace {
struct MdwBufs {
  float* part;
  int32_t* qoff;
  int2* rec;
  int32_t* src;
  int32_t* cnt;
  int32_t* perm;
  int32_t* inv;
};
MdwBufs mdw_bufs(const MdwPlan& p, int N_in, int N_out, int64_t out_cap, void* workspace, float* dW) {
  Carve ws(workspace);
  MdwBufs b{};
  b.part = p.n_chunks > 1 ? ws.take<float>((size_t)p.n_chunks * N_in * (4 * ((N_out + 3) / 4))) : dW;
  b.qoff = ws.take<int32_t>((size_t)p.n_win * kMQLd);
  b.rec = ws.take<int2>((size_t)out_cap + 4);
  b.src = ws.take<int32_t>((size_t)out_cap + 1);
  b.cnt = ws.take<int32_t>((size_t)N_out);
  b.perm = ws.take<int32_t>((size_t)N_out);
  b.inv = ws.take<int32_t>((size_t)N_out + 4);
  return b;
}
}  // namespace

void mdw_enqueue_layout(int T, int B, int N_in, int N_out, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                        int64_t out_cap, void* workspace, hipStream_t s) {
  const MdwPlan p = plan_mdw(T, B, N_in, N_out);
  const MdwBufs b = mdw_bufs(p, N_in, N_out, out_cap, workspace, nullptr);
  hipLaunchKernelGGL(mdw_zero, dim3(1), dim3(256), 0, s, b.cnt, N_out);
  const int cblocks = std::max(1, std::min(cu_count(), (int)((out_cap + 4095) / 4096)));
  hipLaunchKernelGGL(mdw_colcount, dim3((unsigned)cblocks), dim3(256), 0, s, T * B, N_out, out_row_ptr, out_col_idx,
                     out_cap, b.cnt);
  hipLaunchKernelGGL(mdw_perm, dim3((unsigned)((N_out + kWave - 1) / kWave)), dim3(kPermWaves * kWave), 0, s, N_out, b.cnt,
                     b.perm, b.inv);
  hipLaunchKernelGGL(mdw_layout, dim3((unsigned)p.n_win), dim3(kLayWaves * kWave), 0, s, T * B, N_out, out_row_ptr,
                     out_col_idx, out_cap, b.perm, b.qoff, b.rec, b.src);
}

void mdw_enqueue_rest(const float* trace_in, int T, int B, int N_in, int N_out, const float* out_g, const float* eps_out,
                      int64_t out_cap, float* dW, void* workspace, hipStream_t s) {
  const MdwPlan p = plan_mdw(T, B, N_in, N_out);
  const MdwBufs b = mdw_bufs(p, N_in, N_out, out_cap, workspace, dW);
  hipLaunchKernelGGL(mdw_gate, dim3((unsigned)p.n_win), dim3(256), 0, s, b.qoff, out_cap, b.src, out_g, eps_out, b.rec);
  ensure_dynamic_lds((const void*)mdw_kernel, 2 * kMBuf);
  hipLaunchKernelGGL(mdw_kernel, dim3((unsigned)(p.n_itiles * p.n_chunks)), dim3(kMThreads), 2 * kMBuf, s, trace_in,
                     T * B, N_in, N_out, b.qoff, b.rec, b.inv, out_cap, p.n_win, p.n_itiles, b.part,
                     p.n_chunks > 1);
  if (p.n_chunks > 1) {
    const int S = 4 * ((N_out + 3) / 4);
    const int64_t n = (int64_t)N_in * S;
    hipLaunchKernelGGL(mdw_reduce, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, b.part, p.n_chunks, N_in, N_out,
                       S, b.inv, dW);
  }
}

}  // namespace snn
