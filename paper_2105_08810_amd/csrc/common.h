// Shared host/device helpers of libsnn (internal header).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "../../include/snn.h"

namespace snn {

constexpr int kWave = 64;  // CDNA4 wavefront width

// ------------------------------------------------------------------ host-side checks

inline bool bad_dim(int x) { return x <= 0; }

// Element count of a [T,B,N] tensor must stay below 2^31 (int32 CSR offsets and indexing).
inline bool too_big(int T, int B, int N) {
  return (int64_t)T * (int64_t)B * (int64_t)N >= ((int64_t)1 << 31);
}

inline bool bad_alpha(float a) { return !(a > 0.0f && a <= 1.0f); }  // also rejects NaN

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline snn_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? SNN_OK : SNN_ERR_HIP;
}

// Bump allocator over the caller's workspace.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* p) : base(static_cast<char*>(p)) {}
  template <class T>
  T* take(size_t n) {
    T* p = reinterpret_cast<T*>(base ? base + off : nullptr);
    off += align256(n * sizeof(T));
    return p;
  }
};

// Number of compute units of the current device (cached per process and device).
int cu_count();

// Raises a kernel's dynamic-LDS limit on the current device to at least `bytes`. The attribute
// is set once per device, kernel and size and remembered (thread-safe); later calls only look up.
void ensure_dynamic_lds(const void* kernel, int bytes);

// Sparse dW on the matrix cores (dw_mfma.hip), for 512 <= N_out <= 1024, N_in % 4 == 0 and at most
// 10% of the entries active.
struct MdwPlan {
  int n_win, n_itiles, n_chunks, wpc;  // windows of rows, input tiles, chunks of windows, windows per chunk
};
bool mdw_eligible(int T, int B, int N_in, int N_out, int64_t out_cap);
MdwPlan plan_mdw(int T, int B, int N_in, int N_out);
size_t mdw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap);
// Structure-only part: sorts each window's entries by column quad into the workspace.
void mdw_enqueue_layout(int T, int B, int N_in, int N_out, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                        int64_t out_cap, void* workspace, hipStream_t s);
// The rest (needs eps): G into the sorted entries, the accumulation, the chunk reduction into dW.
void mdw_enqueue_rest(const float* trace_in, int T, int B, int N_in, int N_out, const float* out_g, const float* eps_out,
                      int64_t out_cap, float* dW, void* workspace, hipStream_t s);

// Exclusive scan of counts[0..n) into out[0..n] (out[n] = total) and *total64 = total.
// temp must hold scan_temp_elems(n) int32 values.
size_t scan_temp_elems(int n);
void launch_exclusive_scan(const int32_t* counts, int n, int32_t* out, int64_t* total64, int32_t* temp,
                           hipStream_t stream);

// ------------------------------------------------------------------ device helpers

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Lanes below the calling lane that have bits set in mask.
__device__ __forceinline__ int mask_prefix(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Inclusive prefix over the wave's lanes.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int u = __shfl_up(v, off, kWave);
    if (l >= off) v += u;
  }
  return v;
}

}  // namespace snn
