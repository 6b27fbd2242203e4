// Active-set compaction (Definition 1) into CSR, with the truncated spike derivative
// g(V) = 1/(beta |V - theta| + 1)^2 at each active entry (Definition 2; surrogate of Sec. 3).
//
// Three passes over rows r = t*B + b of V [T*B, N]; V is read once unless a row holds more
// than kStage active entries:
//   count  one wavefront per row: predicate per element, wave ballot + lane prefix (mbcnt)
//          give each active element its rank in the row; the first kStage (column, g) pairs are
//          staged in the workspace and the row's count is written
//   scan   device-wide exclusive scan -> row_ptr, nnz
//   fill   one wavefront per row copies the staged pairs to their CSR slots (col_idx stays
//          ascending inside a row); a row with more than kStage entries is re-read from V for
//          the rest. Entries at slots >= capacity are dropped.
// The predicate |V - theta| < b_th is evaluated in float32 exactly as written (one rounded
// subtraction, then fabs and a strict compare), so the integer outputs are bit-exact.
#include "common.h"

#include <mutex>

namespace snn {
namespace {

constexpr int kRowsPerBlock = 4;  // one wavefront per row
constexpr int kThreads = kRowsPerBlock * kWave;
constexpr int kStage = 64;  // staged entries per row
constexpr int kGroup = 4;   // 256-wide slices of a row loaded together

struct Staged {
  int32_t j;
  float g;
};

__device__ __forceinline__ bool is_active(float v, float theta, float bth) { return fabsf(v - theta) < bth; }

__device__ __forceinline__ float surrogate(float v, float theta, float beta) {
  const float x = __fadd_rn(__fmul_rn(beta, fabsf(v - theta)), 1.0f);
  return 1.0f / __fmul_rn(x, x);
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void compact_count(const float* __restrict__ V, int rows, int N, float theta,
                                                          float bth, float beta, int32_t* __restrict__ counts,
                                                          Staged* __restrict__ stage, int scap) {
  const int l = lane_id();
  const int r = blockIdx.x * kRowsPerBlock + (int)(threadIdx.x / kWave);
  if (r >= rows) return;
  const float* row = V + (size_t)r * N;
  Staged* st = stage + (size_t)r * scap;
  int base = 0;
  if (VEC) {
    // lane l holds elements 4l..4l+3 of each 256-wide slice; ascending order is (lane, q). The
    // slices of a 1024-wide group are loaded together before any is used.
    for (int g0 = 0; g0 < N; g0 += kGroup * 4 * kWave) {
      float4 v[kGroup];
#pragma unroll
      for (int c = 0; c < kGroup; ++c) {
        const int j = g0 + c * 4 * kWave + 4 * l;
        v[c] = j < N ? *reinterpret_cast<const float4*>(row + j) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int c = 0; c < kGroup; ++c) {
        const int j = g0 + c * 4 * kWave + 4 * l;
        const float vv[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
        bool a[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) a[q] = (j < N) && is_active(vv[q], theta, bth);
        const uint64_t m0 = __ballot(a[0]), m1 = __ballot(a[1]), m2 = __ballot(a[2]), m3 = __ballot(a[3]);
        int pos = base + mask_prefix(m0) + mask_prefix(m1) + mask_prefix(m2) + mask_prefix(m3);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (a[q]) {
            if (pos < scap) st[pos] = Staged{j + q, surrogate(vv[q], theta, beta)};
            ++pos;
          }
        }
        base += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
      }
    }
  } else {
    for (int j0 = 0; j0 < N; j0 += kWave) {
      const int j = j0 + l;
      const float v = j < N ? row[j] : 0.0f;
      const bool a = (j < N) && is_active(v, theta, bth);
      const uint64_t m = __ballot(a);
      const int pos = base + mask_prefix(m);
      if (a && pos < scap) st[pos] = Staged{j, surrogate(v, theta, beta)};
      base += __popcll(m);
    }
  }
  if (l == 0) counts[r] = base;
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void compact_fill(const float* __restrict__ V, int rows, int N, float theta,
                                                         float bth, float beta, const int32_t* __restrict__ row_ptr,
                                                         const Staged* __restrict__ stage, int scap,
                                                         int32_t* __restrict__ col_idx, float* __restrict__ g_act,
                                                         int64_t cap) {
  const int l = lane_id();
  const int r = blockIdx.x * kRowsPerBlock + (int)(threadIdx.x / kWave);
  if (r >= rows) return;
  const int64_t dst = row_ptr[r];
  const int cnt = row_ptr[r + 1] - row_ptr[r];
  const Staged* st = stage + (size_t)r * scap;
  for (int k = l; k < min(cnt, scap); k += kWave) {
    const Staged x = st[k];
    if (dst + k < cap) {
      col_idx[dst + k] = x.j;
      if (g_act) g_act[dst + k] = x.g;
    }
  }
  if (cnt <= scap) return;
  // more active entries than staged: walk the row again and place ranks >= scap
  const float* row = V + (size_t)r * N;
  int base = 0;
  if (VEC) {
    for (int j0 = 0; j0 < N; j0 += 4 * kWave) {
      const int j = j0 + 4 * l;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (j < N) v = *reinterpret_cast<const float4*>(row + j);
      const float vv[4] = {v.x, v.y, v.z, v.w};
      bool a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = (j < N) && is_active(vv[q], theta, bth);
      const uint64_t m0 = __ballot(a[0]), m1 = __ballot(a[1]), m2 = __ballot(a[2]), m3 = __ballot(a[3]);
      int pos = base + mask_prefix(m0) + mask_prefix(m1) + mask_prefix(m2) + mask_prefix(m3);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (a[q]) {
          if (pos >= scap && dst + pos < cap) {
            col_idx[dst + pos] = j + q;
            if (g_act) g_act[dst + pos] = surrogate(vv[q], theta, beta);
          }
          ++pos;
        }
      }
      base += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
    }
  } else {
    for (int j0 = 0; j0 < N; j0 += kWave) {
      const int j = j0 + l;
      const float v = j < N ? row[j] : 0.0f;
      const bool a = (j < N) && is_active(v, theta, bth);
      const uint64_t m = __ballot(a);
      const int pos = base + mask_prefix(m);
      if (a && pos >= scap && dst + pos < cap) {
        col_idx[dst + pos] = j;
        if (g_act) g_act[dst + pos] = surrogate(v, theta, beta);
      }
      base += __popcll(m);
    }
  }
}

// ------------------------------------------------------------------ from a bitset
// Bit (t, k), k = b * N + j, of word t * W64 + k / 64 (W64 = ceil(B N / 64)) marks an active
// entry (as snn_lif_forward_active writes it). Window w of row (t, b) = row bits [64 w, 64 w + 64).
__device__ __forceinline__ uint64_t row_window(const uint64_t* __restrict__ bits, size_t W64, int t, size_t bN,
                                               int N, int w) {
  const size_t bit0 = bN + (size_t)kWave * w;
  const size_t wi = bit0 / kWave;
  const int sh = (int)(bit0 % kWave);
  const uint64_t* row = bits + (size_t)t * W64;
  uint64_t x = row[wi] >> sh;
  if (sh) x |= (wi + 1 < W64 ? row[wi + 1] : 0ull) << (kWave - sh);
  const int rem = N - kWave * w;
  if (rem < kWave) x &= (1ull << rem) - 1ull;
  return x;
}

// Count and fill run over tiles of TR consecutive rows, one 1024-thread block per tile: the count
// kernel writes every row's count and the tile's total; the fill kernel forms its tile's row
// pointers itself (the totals of the tiles before it, at most kMaxTiles of them, plus a block
// scan of its rows' counts), then places the entries. Two kernels instead of count, a
// three-kernel scan and fill. A wavefront takes RPW = 64 / nw rows at a time when a row has
// nw <= 64 windows (lane l: row l / nw of the group, window l % nw), else one row with the windows
// walked 64 at a time; positions inside a row come from a wavefront-wide inclusive scan minus its
// value just before the row's first lane.
constexpr int kTileThreads = 1024;
constexpr int kTileWaves = kTileThreads / kWave;
constexpr int kMaxTiles = 4096;

struct TilePlan {
  int tr, n_tiles, rpw;
};

// Tiles of 64 rows (long rows, one per wavefront: 16), doubled until there are at most 1024
// tiles (long rows: kMaxTiles). Measured: fewer, longer tiles cost more in the fill's V gathers
// than the shorter sum over earlier tiles saves, except for long rows.
TilePlan plan_tiles(int rows, int N) {
  TilePlan p{};
  const int nw = (N + kWave - 1) / kWave;
  p.rpw = nw <= kWave ? kWave / nw : 1;
  p.tr = p.rpw > 1 ? 64 : kTileWaves;
  const int max_tiles = p.rpw > 1 ? 1024 : kMaxTiles;
  while ((rows + p.tr - 1) / p.tr > max_tiles) p.tr *= 2;
  p.n_tiles = (rows + p.tr - 1) / p.tr;
  return p;
}

__global__ __launch_bounds__(kTileThreads) void bits_count(const uint64_t* __restrict__ bits, int T, int B, int N,
                                                           int tr, int rpw, int32_t* __restrict__ counts,
                                                           int32_t* __restrict__ tile_sum) {
  __shared__ int wsum[kTileWaves];
  const int l = lane_id();
  const int wv = threadIdx.x / kWave;
  const int rows = T * B;
  const int nw = (N + kWave - 1) / kWave;
  const size_t W64 = ((size_t)B * N + kWave - 1) / kWave;
  const int t0 = blockIdx.x * tr, t1 = min(rows, t0 + tr);
  int total = 0;
  for (int r0 = t0 + wv * rpw; r0 < t1; r0 += kTileWaves * rpw) {
    if (rpw > 1) {
      const int k = l / nw, w = l - k * nw;
      const int r = r0 + k;
      const bool ok = k < rpw && r < t1;
      const int c = ok ? __popcll(row_window(bits, W64, r / B, (size_t)(r % B) * N, N, w)) : 0;
      const int incl = wave_incl_scan(c);
      const int first = k * nw;  // lane of the row's first window
      const int before = __shfl(incl, max(first - 1, 0), kWave);  // every lane takes part in the exchange
      if (ok && w == nw - 1) counts[r] = incl - (first > 0 ? before : 0);
      total += __shfl(incl, kWave - 1, kWave);
    } else {
      int c = 0;
      for (int w0 = 0; w0 < nw; w0 += kWave)
        if (w0 + l < nw) c += __popcll(row_window(bits, W64, r0 / B, (size_t)(r0 % B) * N, N, w0 + l));
      c = wave_sum_int(c);
      if (l == 0) counts[r0] = c;
      total += c;
    }
  }
  if (l == 0) wsum[wv] = total;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int k = 0; k < kTileWaves; ++k) s += wsum[k];
    tile_sum[blockIdx.x] = s;
  }
}

// Places a lane's set bits of one window at pos, pos + 1, ... (up to four V loads in flight).
__device__ __forceinline__ void place_window(uint64_t x, int jbase, int64_t pos, const float* __restrict__ vrow,
                                             float theta, float beta, int32_t* __restrict__ col_idx,
                                             float* __restrict__ g_act, int64_t cap) {
  while (__ballot(x != 0ull)) {
    int jj[4];
    float vv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      jj[u] = x ? jbase + (__ffsll((long long)x) - 1) : -1;
      x &= x - 1ull;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) vv[u] = (g_act && jj[u] >= 0) ? vrow[jj[u]] : 0.0f;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (jj[u] >= 0) {
        if (pos < cap) {
          col_idx[pos] = jj[u];
          if (g_act) g_act[pos] = surrogate(vv[u], theta, beta);
        }
        ++pos;
      }
    }
  }
}

// tr <= kTileThreads * kMaxPerThread rows per tile.
constexpr int kMaxPerThread = 8;

__global__ __launch_bounds__(kTileThreads) void bits_fill(const uint64_t* __restrict__ bits, const float* __restrict__ V,
                                                          int T, int B, int N, int tr, int rpw, float theta, float beta,
                                                          const int32_t* __restrict__ counts,
                                                          const int32_t* __restrict__ tile_sum,
                                                          int32_t* __restrict__ row_ptr, int64_t* __restrict__ nnz,
                                                          int32_t* __restrict__ col_idx, float* __restrict__ g_act,
                                                          int64_t cap) {
  extern __shared__ int rp_tile[];  // [tr + 1]: the tile's row pointers
  __shared__ int red[kTileWaves];
  __shared__ int base_s;
  const int l = lane_id();
  const int wv = threadIdx.x / kWave;
  const int rows = T * B;
  const int t0 = blockIdx.x * tr, t1 = min(rows, t0 + tr);
  // the totals of the tiles before this one (fixed order: per thread, then the wavefronts in order)
  int p = 0;
  for (int k = threadIdx.x; k < (int)blockIdx.x; k += kTileThreads) p += tile_sum[k];
  p = wave_sum_int(p);
  if (l == 0) red[wv] = p;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int k = 0; k < kTileWaves; ++k) s += red[k];
    base_s = s;
  }
  __syncthreads();
  const int base = base_s;
  // exclusive scan of the tile's row counts; thread x owns rows t0 + x * per .. + per - 1
  const int per = (tr + kTileThreads - 1) / kTileThreads;
  int c[kMaxPerThread];
  int mine = 0;
#pragma unroll
  for (int u = 0; u < kMaxPerThread; ++u) {
    const int r = t0 + threadIdx.x * per + u;
    c[u] = (u < per && r < t1) ? counts[r] : 0;
    mine += c[u];
  }
  const int incl = wave_incl_scan(mine);
  __syncthreads();  // red is reused
  if (l == kWave - 1) red[wv] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < kTileWaves; ++k) {
    const int v = red[k];
    before += k < wv ? v : 0;
    all += v;
  }
  int run = before + incl - mine;
#pragma unroll
  for (int u = 0; u < kMaxPerThread; ++u) {
    const int rl = threadIdx.x * per + u;
    if (u < per && t0 + rl < t1) {
      rp_tile[rl] = base + run;
      row_ptr[t0 + rl] = base + run;
    }
    run += c[u];
  }
  if (threadIdx.x == 0) {
    rp_tile[t1 - t0] = base + all;
    if (t1 == rows) {  // the last tile closes the row pointers and reports the true count
      row_ptr[rows] = base + all;
      *nnz = (int64_t)base + all;
    }
  }
  __syncthreads();
  if (cap <= 0) return;
  const int nw = (N + kWave - 1) / kWave;
  const size_t W64 = ((size_t)B * N + kWave - 1) / kWave;
  for (int r0 = t0 + wv * rpw; r0 < t1; r0 += kTileWaves * rpw) {
    if (rpw > 1) {
      const int k = l / nw, w = l - k * nw;
      const int r = r0 + k;
      const bool ok = k < rpw && r < t1;
      const uint64_t x = ok ? row_window(bits, W64, r / B, (size_t)(r % B) * N, N, w) : 0ull;
      const int64_t dst = ok ? rp_tile[r - t0] : 0;
      const int cw = __popcll(x);
      const int in = wave_incl_scan(cw);
      const int first = k * nw;
      const int prev = __shfl(in, max(first - 1, 0), kWave);  // every lane takes part in the exchange
      const int bef = first > 0 ? prev : 0;
      place_window(x, kWave * w, dst + (in - cw - bef), V + (size_t)(ok ? r : 0) * N, theta, beta, col_idx, g_act,
                   cap);
    } else {
      const int r = r0;
      const float* vrow = V + (size_t)r * N;
      int64_t b0 = rp_tile[r - t0];
      for (int w0 = 0; w0 < nw; w0 += kWave) {
        const int w = w0 + l;
        const uint64_t x = w < nw ? row_window(bits, W64, r / B, (size_t)(r % B) * N, N, w) : 0ull;
        const int cw = __popcll(x);
        const int in = wave_incl_scan(cw);
        place_window(x, kWave * w, b0 + in - cw, vrow, theta, beta, col_idx, g_act, cap);
        b0 += __shfl(in, kWave - 1, kWave);
      }
    }
  }
}

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" size_t snn_active_compact_workspace(int T, int B, int N) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return 0;
  const int rows = T * B;
  Carve c(nullptr);
  c.take<int32_t>(rows);
  c.take<int32_t>(scan_temp_elems(rows));
  c.take<Staged>((size_t)rows * std::min(N, kStage));
  return c.off;
}

extern "C" snn_status snn_active_compact(const float* V, int T, int B, int N, float theta, float b_th, float beta,
                                         int32_t* row_ptr, int32_t* col_idx, float* g_act, int64_t capacity,
                                         int64_t* nnz_dev, void* workspace, size_t workspace_bytes, void* stream) {
  if (!V || !row_ptr || !nnz_dev || !workspace) return SNN_ERR_INVALID_ARG;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return SNN_ERR_INVALID_ARG;
  if (isnan(theta) || isnan(b_th) || b_th < 0.0f || isnan(beta) || beta < 0.0f) return SNN_ERR_INVALID_ARG;
  if (capacity < 0 || (capacity > 0 && !col_idx)) return SNN_ERR_INVALID_ARG;
  if (workspace_bytes < snn_active_compact_workspace(T, B, N)) return SNN_ERR_INVALID_ARG;

  hipStream_t s = static_cast<hipStream_t>(stream);
  const int rows = T * B;
  Carve ws(workspace);
  int32_t* counts = ws.take<int32_t>(rows);
  int32_t* temp = ws.take<int32_t>(scan_temp_elems(rows));
  const int scap = std::min(N, kStage);
  Staged* stage = ws.take<Staged>((size_t)rows * scap);
  const bool vec = (N % 4) == 0 && (reinterpret_cast<uintptr_t>(V) % 16) == 0;
  const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock);
  if (vec)
    hipLaunchKernelGGL(compact_count<true>, grid, dim3(kThreads), 0, s, V, rows, N, theta, b_th, beta, counts, stage,
                       scap);
  else
    hipLaunchKernelGGL(compact_count<false>, grid, dim3(kThreads), 0, s, V, rows, N, theta, b_th, beta, counts,
                       stage, scap);
  launch_exclusive_scan(counts, rows, row_ptr, nnz_dev, temp, s);
  if (capacity > 0) {
    if (vec)
      hipLaunchKernelGGL(compact_fill<true>, grid, dim3(kThreads), 0, s, V, rows, N, theta, b_th, beta, row_ptr,
                         stage, scap, col_idx, g_act, capacity);
    else
      hipLaunchKernelGGL(compact_fill<false>, grid, dim3(kThreads), 0, s, V, rows, N, theta, b_th, beta, row_ptr,
                         stage, scap, col_idx, g_act, capacity);
  }
  return launch_status();
}

extern "C" size_t snn_active_compact_bits_workspace(int T, int B, int N) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return 0;
  const int rows = T * B;
  const TilePlan p = plan_tiles(rows, N);
  Carve c(nullptr);
  c.take<int32_t>(rows);
  c.take<int32_t>(p.n_tiles);
  return c.off;
}

namespace snn {
namespace {

// Validation shared by snn_active_compact_bits and its allocation-free form.
bool compact_bits_args_ok(const uint64_t* active_bits, const float* V, int T, int B, int N, float theta, float beta,
                          const int32_t* row_ptr, const int32_t* col_idx, const float* g_act, int64_t capacity,
                          const int64_t* nnz_dev) {
  if (!active_bits || !row_ptr || !nnz_dev) return false;
  if (bad_dim(T) || bad_dim(B) || bad_dim(N) || too_big(T, B, N)) return false;
  if (isnan(theta) || isnan(beta) || beta < 0.0f) return false;
  if (capacity < 0 || (capacity > 0 && !col_idx) || (g_act && !V)) return false;
  return true;
}

// The count, scan and fill passes, with the row counts and scan temporaries in `workspace`
// (at least snn_active_compact_bits_workspace bytes; every byte used is written before it is
// read, so it needs no clearing).
snn_status enqueue_compact_bits(const uint64_t* active_bits, const float* V, int T, int B, int N, float theta,
                                float beta, int32_t* row_ptr, int32_t* col_idx, float* g_act, int64_t capacity,
                                int64_t* nnz_dev, void* workspace, hipStream_t s) {
  const int rows = T * B;
  const TilePlan p = plan_tiles(rows, N);
  if (p.tr > kTileThreads * kMaxPerThread) return SNN_ERR_UNSUPPORTED;  // more than 8 M rows
  Carve ws(workspace);
  int32_t* counts = ws.take<int32_t>(rows);
  int32_t* tsum = ws.take<int32_t>(p.n_tiles);
  hipLaunchKernelGGL(bits_count, dim3((unsigned)p.n_tiles), dim3(kTileThreads), 0, s, active_bits, T, B, N, p.tr, p.rpw,
                     counts, tsum);
  hipLaunchKernelGGL(bits_fill, dim3((unsigned)p.n_tiles), dim3(kTileThreads), (size_t)(p.tr + 1) * sizeof(int), s,
                     active_bits, V, T, B, N, p.tr, p.rpw, theta, beta, counts, tsum, row_ptr, nnz_dev, col_idx, g_act,
                     capacity);
  return launch_status();
}

}  // namespace
}  // namespace snn

extern "C" snn_status snn_active_compact_bits(const uint64_t* active_bits, const float* V, int T, int B, int N,
                                              float theta, float beta, int32_t* row_ptr, int32_t* col_idx,
                                              float* g_act, int64_t capacity, int64_t* nnz_dev, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  if (!workspace) return SNN_ERR_INVALID_ARG;
  if (!compact_bits_args_ok(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity, nnz_dev))
    return SNN_ERR_INVALID_ARG;
  if (workspace_bytes < snn_active_compact_bits_workspace(T, B, N)) return SNN_ERR_INVALID_ARG;
  return enqueue_compact_bits(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity, nnz_dev,
                              workspace, static_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------------ allocation-free form
//
// The workspace of snn_active_compact_bits_noalloc is a file-scope device array: one copy per
// GPU, part of the code object's memory, held until the process ends. Host code never passes the
// array's name to a kernel (on the host it names a stand-in, not device memory): the device
// address is looked up once per device, with that device current, and kept.
namespace snn {
namespace {

constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device (nullptr if it cannot be had).
void* scratch_on_current_device() {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    addr[dev] = p;
  }
  return addr[dev];
}

}  // namespace
}  // namespace snn

extern "C" snn_status snn_active_compact_bits_noalloc(const uint64_t* active_bits, const float* V, int T, int B,
                                                      int N, float theta, float beta, int32_t* row_ptr,
                                                      int32_t* col_idx, float* g_act, int64_t capacity,
                                                      int64_t* nnz_dev, void* stream) {
  if (!compact_bits_args_ok(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity, nnz_dev))
    return SNN_ERR_INVALID_ARG;
  if (snn_active_compact_bits_workspace(T, B, N) > kNoAllocScratchBytes) return SNN_ERR_UNSUPPORTED;
  void* ws = scratch_on_current_device();
  if (!ws) return SNN_ERR_HIP;
  return enqueue_compact_bits(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity, nnz_dev, ws,
                              static_cast<hipStream_t>(stream));
}
