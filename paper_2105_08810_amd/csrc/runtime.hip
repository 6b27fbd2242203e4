// Status strings, device queries and the device-wide exclusive scan used to turn per-row
// counts into CSR row pointers.
#include "common.h"

#include <mutex>
#include <vector>

extern "C" const char* snn_status_string(int status) {
  switch (status) {
    case SNN_OK: return "SNN_OK";
    case SNN_ERR_INVALID_ARG: return "SNN_ERR_INVALID_ARG";
    case SNN_ERR_UNSUPPORTED: return "SNN_ERR_UNSUPPORTED";
    case SNN_ERR_HIP: return "SNN_ERR_HIP";
    default: return "SNN_UNKNOWN_STATUS";
  }
}

namespace snn {

int cu_count() {
  static int cached_dev = -1;
  static int cached = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev != cached_dev) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached = n;
    cached_dev = dev;
  }
  return cached;
}

void ensure_dynamic_lds(const void* kernel, int bytes) {
  struct Done {
    int dev;
    const void* kernel;
    int bytes;
  };
  static std::mutex mu;
  static std::vector<Done> done;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return;
  std::lock_guard<std::mutex> lock(mu);
  for (const Done& d : done)
    if (d.dev == dev && d.kernel == kernel && d.bytes >= bytes) return;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess)
    done.push_back({dev, kernel, bytes});
}

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 8;
constexpr int kScanTile = kScanThreads * kScanPerThread;
constexpr int kOwnPrefixTiles = 1024;

// Block-wide exclusive scan of one value per thread; returns the block total through *total.
__device__ int block_excl_scan(int v, int* total) {
  __shared__ int wave_tot[kScanThreads / kWave];
  const int l = lane_id();
  const int w = threadIdx.x / kWave;
  int incl = wave_incl_scan(v);
  if (l == kWave - 1) wave_tot[w] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < kScanThreads / kWave; ++k) {
    int t = wave_tot[k];
    if (k < w) before += t;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

__device__ __forceinline__ void load_tile(const int32_t* counts, int n, int base, int* x) {
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    int i = base + k;
    x[k] = i < n ? counts[i] : 0;
  }
}

__global__ __launch_bounds__(kScanThreads) void scan_tile_sums(const int32_t* counts, int n, int32_t* sums) {
  int x[kScanPerThread];
  load_tile(counts, n, blockIdx.x * kScanTile + threadIdx.x * kScanPerThread, x);
  int s = 0;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) s += x[k];
  int total;
  (void)block_excl_scan(s, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// One block scans the tile sums in place (exclusive).
__global__ __launch_bounds__(kScanThreads) void scan_sums(int32_t* sums, int nb) {
  int carry = 0;
  for (int base = 0; base < nb; base += kScanTile) {
    int x[kScanPerThread];
    load_tile(sums, nb, base + threadIdx.x * kScanPerThread, x);
    int s = 0;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) s += x[k];
    int total;
    int ex = block_excl_scan(s, &total) + carry;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      int i = base + threadIdx.x * kScanPerThread + k;
      if (i < nb) sums[i] = ex;
      ex += x[k];
    }
    carry += total;
    __syncthreads();
  }
}

// Each tile's offset is sums[tile] (scanned by scan_sums), or, with own_prefix, the sum of the
// earlier tiles' totals formed by the block itself (few tiles: one kernel less on the chain).
__global__ __launch_bounds__(kScanThreads) void scan_apply(const int32_t* counts, int n, const int32_t* sums,
                                                           int nb, int32_t* out, int64_t* total64, int own_prefix) {
  int x[kScanPerThread];
  const int base = blockIdx.x * kScanTile + threadIdx.x * kScanPerThread;
  load_tile(counts, n, base, x);
  int prefix;
  if (own_prefix) {
    int p = 0;
    for (int k = threadIdx.x; k < (int)blockIdx.x; k += kScanThreads) p += sums[k];
    int all;
    (void)block_excl_scan(p, &all);
    prefix = all;
  } else {
    prefix = sums[blockIdx.x];
  }
  int s = 0;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) s += x[k];
  int total;
  int ex = block_excl_scan(s, &total) + prefix;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (base + k < n) out[base + k] = ex;
    ex += x[k];
  }
  if ((int)blockIdx.x == nb - 1 && threadIdx.x == 0) {
    int grand = prefix + total;
    out[n] = grand;
    if (total64) *total64 = (int64_t)grand;
  }
}

}  // namespace

size_t scan_temp_elems(int n) { return (size_t)((n + kScanTile - 1) / kScanTile) + 1; }

void launch_exclusive_scan(const int32_t* counts, int n, int32_t* out, int64_t* total64, int32_t* temp,
                           hipStream_t stream) {
  const int nb = (n + kScanTile - 1) / kScanTile;
  // up to kOwnPrefixTiles tiles each block adds the earlier tiles' totals itself (two kernels);
  // beyond, one block scans the tile totals first (three kernels)
  const bool own = nb <= kOwnPrefixTiles;
  hipLaunchKernelGGL(scan_tile_sums, dim3(nb), dim3(kScanThreads), 0, stream, counts, n, temp);
  if (!own) hipLaunchKernelGGL(scan_sums, dim3(1), dim3(kScanThreads), 0, stream, temp, nb);
  hipLaunchKernelGGL(scan_apply, dim3(nb), dim3(kScanThreads), 0, stream, counts, n, temp, nb, out, total64,
                     own ? 1 : 0);
}

}  // namespace snn
