// The convolutional spiking layer's pooling and backward (the convolutional experiment of
// Sec. 3; network details in App. E): 2x2 max pooling of its spikes into the readout, the
// pooling's share of the active set, the readout's spike gradient routed back through the
// pooling, and the filter gradient, sparse (at the layer's active entries) and dense.
//
// Layout: channels last. Conv neuron n = (y * W + x) * F + f of N = H * W * F; pooled neuron
// np = (py * (W/2) + px) * F + f of Np = (H/2) * (W/2) * F; rows r = t * B + b. Filters
// Wc [3, 3, C, F], output (y, x) reading input (y + ky - 1, x + kx - 1) (zero padding).
// Pooling: P = OR of the 2x2 window; arg = the window position (0..3, row-major) of the first
// spike, 0 when none; the window's gradient goes to that element.

#include <algorithm>

#include "common.h"

namespace snn {
namespace {

constexpr int kCdwThreads = 256;  // dense filter gradient
constexpr int kCdwWaves = kCdwThreads / kWave;
constexpr int kCsdThreads = 1024;  // sparse filter gradient: 16 wavefronts share a block's accumulator
constexpr int kCsdWaves = kCsdThreads / kWave;
constexpr int kCdwMaxBlocks = 1024;
constexpr int kDenseBlocks = 8192;  // blocks of the dense filter gradient (each walks its positions)
constexpr int kDenseMaxC = 4;  // input channels per register group of the dense filter gradient
constexpr int kDenseBatch = 4;  // positions (one channel) per wavefront whose loads are in flight together

unsigned stream_blocks(int64_t items) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 65536));
}

// Rows r = t * B + b run along grid y (grid-stride), pooled neurons of a row along x; with
// VEC (F % 4 == 0) a thread takes four neighbouring filters with 32-bit loads and stores.
template <bool VEC>
__global__ void pool_kernel(const uint8_t* __restrict__ S, int TB, int H, int W, int F, uint8_t* __restrict__ P,
                            uint8_t* __restrict__ arg) {
  const int hw = W / 2;
  const int Np = (H / 2) * hw * F;
  const int N = H * W * F;
  const int j = (blockIdx.x * blockDim.x + threadIdx.x) * (VEC ? 4 : 1);
  if (j >= Np) return;
  const int f = j % F;
  const int pp = j / F;
  const int px = pp % hw;
  const int py = pp / hw;
  const int off = ((2 * py) * W + 2 * px) * F + f;
  for (int r = blockIdx.y; r < TB; r += gridDim.y) {
    const uint8_t* s = S + (int64_t)r * N + off;
    const int64_t o = (int64_t)r * Np + j;
    if (VEC) {
      const uint32_t w0 = *reinterpret_cast<const uint32_t*>(s);
      const uint32_t w1 = *reinterpret_cast<const uint32_t*>(s + F);
      const uint32_t w2 = *reinterpret_cast<const uint32_t*>(s + W * F);
      const uint32_t w3 = *reinterpret_cast<const uint32_t*>(s + W * F + F);
      uint32_t pv = 0, av = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool s0 = (w0 >> (8 * q)) & 0xffu, s1 = (w1 >> (8 * q)) & 0xffu;
        const bool s2 = (w2 >> (8 * q)) & 0xffu, s3 = (w3 >> (8 * q)) & 0xffu;
        pv |= (uint32_t)(s0 | s1 | s2 | s3) << (8 * q);
        av |= (uint32_t)(s0 ? 0 : (s1 ? 1 : (s2 ? 2 : (s3 ? 3 : 0)))) << (8 * q);
      }
      *reinterpret_cast<uint32_t*>(P + o) = pv;
      *reinterpret_cast<uint32_t*>(arg + o) = av;
    } else {
      const bool s0 = s[0] != 0;
      const bool s1 = s[F] != 0;
      const bool s2 = s[W * F] != 0;
      const bool s3 = s[W * F + F] != 0;
      P[o] = (uint8_t)(s0 | s1 | s2 | s3);
      arg[o] = (uint8_t)(s0 ? 0 : (s1 ? 1 : (s2 ? 2 : (s3 ? 3 : 0))));
    }
  }
}

// Pooled neuron (t, kp = b * Np + np) is active iff the conv neuron its pooling picked is
// active: one ballot per wavefront and step writes one word of the pooled bitset.
__global__ void route_bits_kernel(const uint64_t* __restrict__ cbits, const uint8_t* __restrict__ arg, int T, int B,
                                  int H, int W, int F, uint64_t* __restrict__ pbits) {
  const int hw = W / 2;
  const int Np = (H / 2) * hw * F;
  const int N = H * W * F;
  const int64_t W64p = ((int64_t)B * Np + kWave - 1) / kWave;
  const int64_t W64c = ((int64_t)B * N + kWave - 1) / kWave;
  const int kp = blockIdx.x * blockDim.x + threadIdx.x;  // kp - lane is a word start
  if ((int64_t)(kp - lane_id()) >= W64p * kWave) return;  // whole wavefront past the last word
  const bool valid = kp < B * Np;
  int64_t kbase = 0;  // conv neuron of window position 0, and the arg offset inside a step
  int ab = 0;
  if (valid) {
    const int b = kp / Np;
    const int j = kp - b * Np;
    const int f = j % F;
    const int pp = j / F;
    const int px = pp % hw;
    const int py = pp / hw;
    kbase = (int64_t)b * N + ((2 * py) * W + 2 * px) * F + f;
    ab = b * Np + j;
  }
  for (int t = blockIdx.y; t < T; t += gridDim.y) {
    bool on = false;
    if (valid) {
      const int a = arg[(int64_t)t * B * Np + ab] & 3;
      const int64_t kc = kbase + ((a >> 1) * W + (a & 1)) * F;
      on = (cbits[t * W64c + (kc >> 6)] >> (kc & 63)) & 1ull;
    }
    const uint64_t m = __ballot(on);
    if (lane_id() == 0) pbits[t * W64p + (kp >> 6)] = m;
  }
}

// 16 bits to every fourth bit of a word: bit i goes to bit 4 i.
__device__ __forceinline__ uint64_t spread16(uint64_t x) {
  x &= 0xFFFFull;
  x = (x | (x << 24)) & 0x000000FF000000FFull;
  x = (x | (x << 12)) & 0x000F000F000F000Full;
  x = (x | (x << 6)) & 0x0303030303030303ull;
  x = (x | (x << 3)) & 0x1111111111111111ull;
  return x;
}

// As route_bits_kernel with four neighbouring pooled neurons per lane (F % 4 == 0; one 32-bit
// load of their pooling choices): a wavefront covers four words, built from four ballots whose
// bits are interleaved (neuron 4 l + q of the wavefront is ballot q's lane l).
__global__ void route_bits4_kernel(const uint64_t* __restrict__ cbits, const uint8_t* __restrict__ arg, int T, int B,
                                   int H, int W, int F, uint64_t* __restrict__ pbits) {
  const int hw = W / 2;
  const int Np = (H / 2) * hw * F;
  const int N = H * W * F;
  const int64_t W64p = ((int64_t)B * Np + kWave - 1) / kWave;
  const int64_t W64c = ((int64_t)B * N + kWave - 1) / kWave;
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  const int l = lane_id();
  const int64_t word0 = (int64_t)(u - l) / 16;  // the wavefront's first word (256 neurons = 4 words)
  if (word0 >= W64p) return;                    // whole wavefront past the last word
  const int kp = 4 * u;
  const bool valid = kp < B * Np;
  int64_t kbase = 0;
  int ab = 0;
  if (valid) {
    const int b = kp / Np;
    const int j = kp - b * Np;
    const int f = j % F;
    const int pp = j / F;
    const int px = pp % hw;
    const int py = pp / hw;
    kbase = (int64_t)b * N + ((2 * py) * W + 2 * px) * F + f;
    ab = b * Np + j;
  }
  for (int t = blockIdx.y; t < T; t += gridDim.y) {
    uint32_t a4 = 0;
    if (valid) a4 = *reinterpret_cast<const uint32_t*>(arg + (int64_t)t * B * Np + ab);
    uint64_t m[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bool on = false;
      if (valid) {
        const int a = (a4 >> (8 * q)) & 3;
        const int64_t kc = kbase + q + ((a >> 1) * W + (a & 1)) * F;
        on = (cbits[t * W64c + (kc >> 6)] >> (kc & 63)) & 1ull;
      }
      m[q] = __ballot(on);
    }
    if (l < 4 && word0 + l < W64p) {
      uint64_t w = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) w |= spread16(m[q] >> (16 * l)) << q;
      pbits[t * W64p + word0 + l] = w;
    }
  }
}

// As route_bits_kernel with sixteen neighbouring pooled neurons per lane (F % 16 == 0, arg
// 16-byte aligned): the 16 neurons share one pixel, so each window position's candidates are one
// 16-bit field of one conv word; the lane loads its 16 pooling choices and the four words at once
// (no load waits on another), selects per neuron, and four lanes OR their fields into one word.
__device__ __forceinline__ uint32_t low_bits_of_bytes(uint32_t x) {  // bit 0 of byte i -> bit i
  return (((x & 0x01010101u) * 0x01020408u) >> 24) & 0xFu;
}

__global__ void route_bits16_kernel(const uint64_t* __restrict__ cbits, const uint8_t* __restrict__ arg, int T, int B,
                                    int H, int W, int F, uint64_t* __restrict__ pbits) {
  const int hw = W / 2;
  const int64_t Np = (int64_t)(H / 2) * hw * F;
  const int64_t N = (int64_t)H * W * F;
  const int64_t BNp = B * Np;
  const int64_t W64p = (BNp + kWave - 1) / kWave;
  const int64_t W64c = (B * N + kWave - 1) / kWave;
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int l = lane_id();
  if ((u - l) * 16 >= BNp) return;  // whole wavefront past the last neuron
  const int64_t kp = 16 * u;
  const bool valid = kp < BNp;
  int64_t cw[4] = {0, 0, 0, 0};  // conv word of each window position, and the field's shift
  int sh[4] = {0, 0, 0, 0};
  if (valid) {
    const int64_t b = kp / Np;
    const int64_t j = kp - b * Np;
    const int64_t f = j % F;
    const int64_t pp = j / F;
    const int64_t px = pp % hw;
    const int64_t py = pp / hw;
    const int64_t base = b * N + ((2 * py) * W + 2 * px) * F + f;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int64_t kc = base + ((a >> 1) * W + (a & 1)) * F;
      cw[a] = kc >> 6;
      sh[a] = (int)(kc & 63);
    }
  }
  const int64_t word = kp >> 6;
  for (int t = blockIdx.y; t < T; t += gridDim.y) {
    uint32_t r = 0;
    if (valid) {
      const uint4 c = *reinterpret_cast<const uint4*>(arg + (int64_t)t * BNp + kp);
      const uint64_t* wt = cbits + (int64_t)t * W64c;
      uint32_t g[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) g[a] = (uint32_t)(wt[cw[a]] >> sh[a]);
      const uint32_t m0 = low_bits_of_bytes(c.x) | low_bits_of_bytes(c.y) << 4 | low_bits_of_bytes(c.z) << 8 |
                          low_bits_of_bytes(c.w) << 12;
      const uint32_t m1 = low_bits_of_bytes(c.x >> 1) | low_bits_of_bytes(c.y >> 1) << 4 |
                          low_bits_of_bytes(c.z >> 1) << 8 | low_bits_of_bytes(c.w >> 1) << 12;
      r = ((g[0] & ~m0 & ~m1) | (g[1] & m0 & ~m1) | (g[2] & ~m0 & m1) | (g[3] & m0 & m1)) & 0xFFFFu;
    }
    uint64_t v = (uint64_t)r << (16 * (l & 3));
    v |= __shfl_xor(v, 1);
    v |= __shfl_xor(v, 2);
    if ((l & 3) == 0 && word < W64p) pbits[(int64_t)t * W64p + word] = v;
  }
}

__global__ void fill_zero_f(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

// One wavefront per row: each pooled entry's gradient goes to the conv entry its pooling
// picked, found by binary search in the conv row (columns ascending). Entries are clamped to
// the capacities; a conv neuron that is not in the conv row receives nothing.
__global__ void scatter_kernel(int TB, int H, int W, int F, const int32_t* __restrict__ prp,
                               const int32_t* __restrict__ pcol, int64_t pcap, const float* __restrict__ eps_p,
                               const uint8_t* __restrict__ arg, const int32_t* __restrict__ crp,
                               const int32_t* __restrict__ ccol, int64_t ccap, float* __restrict__ eps_c) {
  const int Np = (H / 2) * (W / 2) * F;
  const int r = (int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave);
  if (r >= TB) return;
  const int64_t e0 = std::min<int64_t>(std::max(prp[r], 0), pcap);
  const int64_t e1 = std::min<int64_t>(std::max(prp[r + 1], 0), pcap);
  const int64_t c0 = std::min<int64_t>(std::max(crp[r], 0), ccap);
  const int64_t c1 = std::min<int64_t>(std::max(crp[r + 1], 0), ccap);
  for (int64_t e = e0 + lane_id(); e < e1; e += kWave) {
    const int np_ = pcol[e];
    if ((unsigned)np_ >= (unsigned)Np) continue;
    const int f = np_ % F;
    const int pp = np_ / F;
    const int px = pp % (W / 2);
    const int py = pp / (W / 2);
    const int a = arg[(int64_t)r * Np + np_] & 3;
    const int n = ((2 * py + (a >> 1)) * W + 2 * px + (a & 1)) * F + f;
    int64_t lo = c0, hi = c1;  // first position with col >= n
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (ccol[mid] < n) lo = mid + 1;
      else hi = mid;
    }
    if (lo < c1 && ccol[lo] == n) eps_c[lo] = eps_p[e];
  }
}

// Dense form: eps_c[t,b,y,x,f] = eps_p[t,b,y/2,x/2,f] where (y, x) is the picked element, else 0.
// Rows along grid y (grid-stride), conv neurons of a row along x.
template <bool VEC>
__global__ void scatter_dense_kernel(const float* __restrict__ eps_p, const uint8_t* __restrict__ arg, int TB, int H,
                                     int W, int F, float* __restrict__ eps_c) {
  const int Np = (H / 2) * (W / 2) * F;
  const int N = H * W * F;
  const int n = (blockIdx.x * blockDim.x + threadIdx.x) * (VEC ? 4 : 1);  // VEC: four filters of one pixel
  if (n >= N) return;
  const int f = n % F;
  const int pix = n / F;
  const int y = pix / W;
  const int x = pix - y * W;
  const int jp = ((y / 2) * (W / 2) + x / 2) * F + f;
  const int pos = (y & 1) * 2 + (x & 1);
  for (int r = blockIdx.y; r < TB; r += gridDim.y) {
    const int64_t ip = (int64_t)r * Np + jp;
    if (VEC) {
      const uint32_t a4 = *reinterpret_cast<const uint32_t*>(arg + ip);
      const float4 e4 = *reinterpret_cast<const float4*>(eps_p + ip);
      float4 o;
      o.x = (int)(a4 & 3u) == pos ? e4.x : 0.0f;
      o.y = (int)((a4 >> 8) & 3u) == pos ? e4.y : 0.0f;
      o.z = (int)((a4 >> 16) & 3u) == pos ? e4.z : 0.0f;
      o.w = (int)((a4 >> 24) & 3u) == pos ? e4.w : 0.0f;
      *reinterpret_cast<float4*>(eps_c + (int64_t)r * N + n) = o;
    } else {
      eps_c[(int64_t)r * N + n] = (int)(arg[ip] & 3) == pos ? eps_p[ip] : 0.0f;
    }
  }
}

// Parameters of the pooled form of the sparse filter gradient.
struct PooledArgs {
  const float* V;      // conv layer's V [T*B][H*W*F]
  const uint8_t* arg;  // pooling's pick [T*B][(H/2)*(W/2)*F]
  float theta, b_th, beta;
};

// Surrogate derivative, with the float32 operations of the compaction (no contraction).
__device__ __forceinline__ float surrogate_g(float v, float theta, float beta) {
  const float x = __fadd_rn(__fmul_rn(beta, fabsf(v - theta)), 1.0f);
  return 1.0f / __fmul_rn(x, x);
}

// Sparse filter gradient: blocks take contiguous row ranges, wavefronts rows, lanes the row's
// entries; an entry with G = eps * g != 0 adds G * trace over its 3x3xC input patch into the
// block's float64 accumulator [9 * C][F] in LDS. Each block writes its sums; a fixed-order
// reduction over blocks gives dWc. POOLED: the entries are the pooled CSR's, each standing for
// the conv neuron its pooling picked (window position arg), with G = eps_pooled * g(V) there
// (zero outside the band).
template <int CT, bool POOLED>  // CT > 0: C == CT and the patch's loads are issued together; 0: any C
__global__ __launch_bounds__(kCsdThreads) void conv_dw_sparse_kernel(
    const float* __restrict__ trace, int TB, int H, int W, int C, int F, const int32_t* __restrict__ rp,
    const int32_t* __restrict__ col, const float* __restrict__ g, const float* __restrict__ eps, int64_t cap,
    int rows_per_block, double* __restrict__ part, PooledArgs pa) {
  extern __shared__ double cacc[];  // [9 * C * F]
  const int nacc = 9 * C * F;
  for (int i = threadIdx.x; i < nacc; i += kCsdThreads) cacc[i] = 0.0;
  __syncthreads();
  const int N = H * W * F;
  const int r_lo = blockIdx.x * rows_per_block;
  const int r_hi = min(TB, r_lo + rows_per_block);
  const int w = threadIdx.x / kWave;
  for (int r = r_lo + w; r < r_hi; r += kCsdWaves) {
    const int64_t e0 = std::min<int64_t>(std::max(rp[r], 0), cap);
    const int64_t e1 = std::min<int64_t>(std::max(rp[r + 1], 0), cap);
    const float* tr = trace + (int64_t)r * H * W * C;
    for (int64_t e = e0 + lane_id(); e < e1; e += kWave) {
      // the entry's column and gradient loads go out together; a bad column or a zero gradient
      // is masked, not branched on, so the patch loads below are not held back either
      int n;
      float G0;
      if (POOLED) {
        const int Np = (H / 2) * (W / 2) * F;
        const int p = col[e];
        const bool pv = (unsigned)p < (unsigned)Np;
        const int pc = pv ? p : 0;
        const int a = pa.arg[(int64_t)r * Np + pc] & 3;
        const int q = pc / F;
        const int yy = 2 * (q / (W / 2)) + (a >> 1);
        const int xx = 2 * (q % (W / 2)) + (a & 1);
        n = pv ? (yy * W + xx) * F + (pc - q * F) : -1;
        const float v = pa.V[(int64_t)r * N + (pv ? n : 0)];
        G0 = fabsf(v - pa.theta) < pa.b_th ? eps[e] * surrogate_g(v, pa.theta, pa.beta) : 0.0f;
      } else {
        n = col[e];
        G0 = g ? eps[e] * g[e] : eps[e];
      }
      const bool ok = (unsigned)n < (unsigned)N && G0 != 0.0f;
      const int nc = ok ? n : 0;
      const double G = (double)G0;
      const int f = nc % F;
      const int pix = nc / F;
      const int y = pix / W;
      const int x = pix - y * W;
      if (CT > 0) {
        float tv[9 * (CT > 0 ? CT : 1)];
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) {
          const int yy = y + tap / 3 - 1;
          const int xx = x + tap % 3 - 1;
          const bool in = ok && yy >= 0 && yy < H && xx >= 0 && xx < W;
          const float* tp = tr + ((int64_t)(in ? yy : 0) * W + (in ? xx : 0)) * CT;
#pragma unroll
          for (int c = 0; c < CT; ++c) {
            const float v = tp[c];  // in bounds either way: pixel (0, 0) stands in outside the map
            tv[tap * CT + c] = in ? v : 0.0f;
          }
        }
#pragma unroll
        for (int i = 0; i < 9 * (CT > 0 ? CT : 1); ++i)  // a zero trace adds nothing: skipped
          if (tv[i] != 0.0f) atomicAdd(&cacc[i * F + f], G * (double)tv[i]);
      } else if (ok) {
        for (int ky = 0; ky < 3; ++ky) {
          const int yy = y + ky - 1;
          if (yy < 0 || yy >= H) continue;
          for (int kx = 0; kx < 3; ++kx) {
            const int xx = x + kx - 1;
            if (xx < 0 || xx >= W) continue;
            const float* tp = tr + ((int64_t)yy * W + xx) * C;
            for (int c = 0; c < C; ++c) atomicAdd(&cacc[((ky * 3 + kx) * C + c) * F + f], G * (double)tp[c]);
          }
        }
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nacc; i += kCsdThreads) part[(int64_t)blockIdx.x * nacc + i] = cacc[i];
}

// out[i] = sum over p of part[p][i]: one block per output, 256 threads take fixed strided
// subsets of the partials and a fixed tree joins them (deterministic).
__global__ __launch_bounds__(256) void reduce_parts(const double* __restrict__ part, int n_parts, int n,
                                                    float* __restrict__ out) {
  __shared__ double red[256];
  const int i = blockIdx.x;
  double s = 0.0;
  for (int p = threadIdx.x; p < n_parts; p += 256) s += part[(int64_t)p * n + i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[i] = (float)red[0];
}

// Dense filter gradient of the full (b_th = inf) or truncated surrogate: every position
// (t, b, y, x) and filter f. Lane = filter (F <= 64 per wavefront pass), wavefronts take
// positions; G = eps * g(V) * [|V - theta| < b_th] and the patch's trace values (uniform across
// the wavefront) go into 9 * C float32 registers per lane; blocks then sum their wavefronts in
// LDS (float64 sums) and write float64 partial sums.
template <int CMAX>
__global__ __launch_bounds__(kCdwThreads) void conv_dw_dense_kernel(
    const float* __restrict__ trace, const float* __restrict__ V, const float* __restrict__ eps, int64_t n_pos,
    int H, int W, int C, int F, float theta, float b_th, float beta, int64_t pos_per_block, double* __restrict__ part) {
  __shared__ float red[kCdwWaves][9 * CMAX][kWave];
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int l = lane_id();
  const int nacc = 9 * C * F;
  const int64_t p_lo = (int64_t)blockIdx.x * pos_per_block;
  const int64_t p_hi = std::min<int64_t>(n_pos, p_lo + pos_per_block);
  for (int f0 = 0; f0 < F; f0 += kWave)
    for (int c0 = 0; c0 < C; c0 += CMAX) {  // channels in groups of CMAX registers
      const int CG = min(CMAX, C - c0);
      const int f = f0 + l;
      const bool fv = f < F;
      float acc[9 * CMAX];
#pragma unroll
      for (int q = 0; q < 9 * CMAX; ++q) acc[q] = 0.0f;
      const int HW = H * W;
      const int64_t n_rows = n_pos / HW;
      // positions p = r * HW + pix, U = kDenseBatch of them per wavefront at a time (stride
      // kCdwWaves). Their V values and 3x3xCG patches (lane k of the wavefront loads patch value
      // k, 9 CG U <= 64) go out together; eps is read only for lanes in the band; a patch value
      // reaches every lane by a lane read.
      constexpr int U = kDenseBatch / CMAX;
      const int n_pv = 9 * CG;  // patch values per position
      int64_t r = (p_lo + w) / HW;
      int pix = (int)(p_lo + w - r * HW);
      for (int64_t p0 = p_lo + w; p0 < p_hi; p0 += U * kCdwWaves) {
        int64_t ru[U];
        int yu[U], xu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          ru[u] = r;
          yu[u] = pix / W;
          xu[u] = pix - yu[u] * W;
          pix += kCdwWaves;
          while (pix >= HW) {
            pix -= HW;
            ++r;
          }
        }
        float vu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int64_t pu = min(p0 + (int64_t)u * kCdwWaves, p_hi - 1);  // in range; weight 0 past p_hi
          vu[u] = fv ? V[pu * F + f] : 0.0f;
        }
        float pv = 0.0f;  // lane k < n_pv U: value k % n_pv of position k / n_pv's patch
        {
          const int u = l / n_pv;
          const int k = l - u * n_pv;
          const int tap = k / CG;
          const int c = k - tap * CG;
          int64_t rr = 0;
          int yy = -1, xx = -1;
#pragma unroll
          for (int v = 0; v < U; ++v)
            if (v == u) {
              rr = ru[v];
              yy = yu[v] + tap / 3 - 1;
              xx = xu[v] + tap % 3 - 1;
            }
          const bool in = u < U && rr < n_rows && yy >= 0 && yy < H && xx >= 0 && xx < W;
          if (in) pv = trace[(rr * HW + (int64_t)yy * W + xx) * C + c0 + c];
        }
        float Gu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float d = fabsf(vu[u] - theta);
          const float q = beta * d + 1.0f;
          const bool band = fv && p0 + (int64_t)u * kCdwWaves < p_hi && d < b_th;
          const int64_t pu = min(p0 + (int64_t)u * kCdwWaves, p_hi - 1);
          Gu[u] = band ? eps[pu * F + f] / (q * q) : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (__ballot(Gu[u] != 0.0f) == 0ull) continue;
#pragma unroll
          for (int tap = 0; tap < 9; ++tap)
#pragma unroll
            for (int c = 0; c < CMAX; ++c)
              if (c < CG) {
                const float t = __int_as_float(
                    __builtin_amdgcn_readlane(__float_as_int(pv), u * n_pv + tap * CG + c));
                acc[tap * CMAX + c] += Gu[u] * t;
              }
        }
      }
#pragma unroll
      for (int q = 0; q < 9 * CMAX; ++q) red[w][q][l] = acc[q];
      __syncthreads();
      for (int i = threadIdx.x; i < 9 * CG * kWave; i += kCdwThreads) {
        const int tap = i / (CG * kWave);
        const int c = (i / kWave) % CG;
        const int ll = i % kWave;
        if (f0 + ll < F) {
          double s = 0.0;
          for (int ww = 0; ww < kCdwWaves; ++ww) s += (double)red[ww][tap * CMAX + c][ll];
          part[(int64_t)blockIdx.x * nacc + (tap * C + c0 + c) * F + f0 + ll] = s;
        }
      }
      __syncthreads();
    }
}

bool conv_dims_ok(int T, int B, int H, int W, int F) {
  if (bad_dim(T) || bad_dim(B) || bad_dim(H) || bad_dim(W) || bad_dim(F)) return false;
  if ((H & 1) || (W & 1)) return false;  // 2x2 pooling with stride 2
  if ((int64_t)H * W * F >= ((int64_t)1 << 31)) return false;
  return !too_big(T, B, H * W * F);
}

// blocks of the sparse filter gradient: enough to fill the chip, partial sums kept under 64 MB
int cdw_blocks(int TB, int nacc) {
  const int by_mem = (int)std::max<int64_t>(1, ((int64_t)64 << 20) / ((int64_t)nacc * (int64_t)sizeof(double)));
  return std::max(1, std::min(std::min(kCdwMaxBlocks, by_mem), TB));
}

int64_t dense_blocks(int64_t n_pos) { return std::max<int64_t>(1, std::min<int64_t>(kDenseBlocks, (n_pos + 63) / 64)); }

}  // namespace
}  // namespace snn

using namespace snn;

extern "C" snn_status snn_maxpool_spikes(const uint8_t* S, int T, int B, int H, int W, int F, uint8_t* P,
                                         uint8_t* arg, void* stream) {
  if (!S || !P || !arg) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F)) return SNN_ERR_INVALID_ARG;
  const int Np = (H / 2) * (W / 2) * F;
  const int TB = T * B;
  const bool vec = F % 4 == 0 && ((uintptr_t)S & 3u) == 0 && ((uintptr_t)P & 3u) == 0 && ((uintptr_t)arg & 3u) == 0;
  const int per = vec ? 4 : 1;
  const unsigned bx = (unsigned)((Np / per + 255) / 256);
  const unsigned by = (unsigned)std::max(1, std::min(TB, (int)(65536 / bx) + 1));
  if (vec)
    hipLaunchKernelGGL(pool_kernel<true>, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream), S, TB, H, W, F,
                       P, arg);
  else
    hipLaunchKernelGGL(pool_kernel<false>, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream), S, TB, H, W,
                       F, P, arg);
  return launch_status();
}

extern "C" snn_status snn_pool_route_bits(const uint64_t* conv_bits, const uint8_t* arg, int T, int B, int H, int W,
                                          int F, uint64_t* pool_bits, void* stream) {
  if (!conv_bits || !arg || !pool_bits) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F)) return SNN_ERR_INVALID_ARG;
  const int64_t Np = (int64_t)(H / 2) * (W / 2) * F;
  if ((int64_t)B * Np + kWave >= ((int64_t)1 << 31)) return SNN_ERR_INVALID_ARG;
  const int64_t lanes = ((B * Np + kWave - 1) / kWave) * kWave;
  if (F % 16 == 0 && ((uintptr_t)arg & 15u) == 0) {
    const int64_t threads = ((B * Np / 16 + kWave - 1) / kWave) * kWave;
    const unsigned bx = (unsigned)((threads + 255) / 256);
    const unsigned by = (unsigned)std::max(1, std::min(T, (int)(65536 / bx) + 1));
    hipLaunchKernelGGL(route_bits16_kernel, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream), conv_bits,
                       arg, T, B, H, W, F, pool_bits);
  } else if (F % 4 == 0 && ((uintptr_t)arg & 3u) == 0) {
    const int64_t threads = ((B * Np / 4 + kWave - 1) / kWave) * kWave;
    const unsigned bx = (unsigned)((threads + 255) / 256);
    const unsigned by = (unsigned)std::max(1, std::min(T, (int)(65536 / bx) + 1));
    hipLaunchKernelGGL(route_bits4_kernel, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream), conv_bits, arg,
                       T, B, H, W, F, pool_bits);
  } else {
    const unsigned bx = (unsigned)((lanes + 255) / 256);
    const unsigned by = (unsigned)std::max(1, std::min(T, (int)(65536 / bx) + 1));
    hipLaunchKernelGGL(route_bits_kernel, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream), conv_bits, arg,
                       T, B, H, W, F, pool_bits);
  }
  return launch_status();
}

extern "C" snn_status snn_pool_scatter_eps(int T, int B, int H, int W, int F, const int32_t* pool_row_ptr,
                                           const int32_t* pool_col_idx, int64_t pool_cap, const float* eps_pool,
                                           const uint8_t* arg, const int32_t* conv_row_ptr,
                                           const int32_t* conv_col_idx, int64_t conv_cap, float* eps_conv,
                                           void* stream) {
  if (!pool_row_ptr || !arg || !conv_row_ptr || !eps_conv) return SNN_ERR_INVALID_ARG;
  if (pool_cap < 0 || conv_cap < 0) return SNN_ERR_INVALID_ARG;
  if (pool_cap > 0 && (!pool_col_idx || !eps_pool)) return SNN_ERR_INVALID_ARG;
  if (conv_cap > 0 && !conv_col_idx) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (conv_cap == 0) return SNN_OK;
  hipLaunchKernelGGL(fill_zero_f, dim3(stream_blocks(conv_cap)), dim3(256), 0, s, eps_conv, conv_cap);
  const int TB = T * B;
  if (pool_cap > 0)
    hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)(((int64_t)TB * kWave + 255) / 256)), dim3(256), 0, s, TB, H, W,
                       F, pool_row_ptr, pool_col_idx, pool_cap, eps_pool, arg, conv_row_ptr, conv_col_idx, conv_cap,
                       eps_conv);
  return launch_status();
}

extern "C" snn_status snn_pool_scatter_eps_dense(const float* eps_pool, const uint8_t* arg, int T, int B, int H, int W,
                                                 int F, float* eps_conv, void* stream) {
  if (!eps_pool || !arg || !eps_conv) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F)) return SNN_ERR_INVALID_ARG;
  const int N = H * W * F;
  const int TB = T * B;
  const bool vec = F % 4 == 0 && ((uintptr_t)arg & 3u) == 0 && ((uintptr_t)eps_pool & 15u) == 0 &&
                   ((uintptr_t)eps_conv & 15u) == 0;
  const unsigned bx = (unsigned)((N / (vec ? 4 : 1) + 255) / 256);
  const unsigned by = (unsigned)std::max(1, std::min(TB, (int)(65536 / bx) + 1));
  if (vec)
    hipLaunchKernelGGL(scatter_dense_kernel<true>, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream),
                       eps_pool, arg, TB, H, W, F, eps_conv);
  else
    hipLaunchKernelGGL(scatter_dense_kernel<false>, dim3(bx, by), dim3(256), 0, static_cast<hipStream_t>(stream),
                       eps_pool, arg, TB, H, W, F, eps_conv);
  return launch_status();
}

extern "C" size_t snn_conv_sparse_dw_workspace(int T, int B, int H, int W, int C, int F) {
  if (!conv_dims_ok(T, B, H, W, F) || bad_dim(C) || C * F > 2048) return 0;
  return align256((size_t)cdw_blocks(T * B, 9 * C * F) * 9 * C * F * sizeof(double));
}

extern "C" snn_status snn_conv_sparse_dw(const float* trace_in, int T, int B, int H, int W, int C, int F,
                                         const int32_t* conv_row_ptr, const int32_t* conv_col_idx,
                                         const float* conv_g, const float* eps_conv, int64_t conv_cap, float* dWc,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!trace_in || !conv_row_ptr || !dWc || !workspace) return SNN_ERR_INVALID_ARG;
  if (conv_cap < 0 || (conv_cap > 0 && (!conv_col_idx || !eps_conv))) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F) || bad_dim(C) || too_big(T, B, H * W * C)) return SNN_ERR_INVALID_ARG;
  if (C * F > 2048) return SNN_ERR_UNSUPPORTED;  // the block accumulator is 9 * C * F float64 in LDS
  if (workspace_bytes < snn_conv_sparse_dw_workspace(T, B, H, W, C, F)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int TB = T * B;
  const int nb = cdw_blocks(TB, 9 * C * F);
  const int rpb = (TB + nb - 1) / nb;
  const int nacc = 9 * C * F;
  double* part = static_cast<double*>(workspace);
  const size_t lds = (size_t)nacc * sizeof(double);
  const PooledArgs none{nullptr, nullptr, 0.0f, 0.0f, 0.0f};
  auto launch = [&](auto kernel) {
    ensure_dynamic_lds((const void*)kernel, (int)lds);
    hipLaunchKernelGGL(kernel, dim3((unsigned)nb), dim3(kCsdThreads), lds, s, trace_in, TB, H, W, C, F, conv_row_ptr,
                       conv_col_idx, conv_g, eps_conv, conv_cap, rpb, part, none);
  };
  if (C == 1) launch(conv_dw_sparse_kernel<1, false>);
  else if (C == 2) launch(conv_dw_sparse_kernel<2, false>);
  else launch(conv_dw_sparse_kernel<0, false>);
  hipLaunchKernelGGL(reduce_parts, dim3((unsigned)nacc), dim3(256), 0, s, part, nb, nacc, dWc);
  return launch_status();
}

extern "C" snn_status snn_conv_sparse_dw_pooled(const float* trace_in, const float* V, const uint8_t* arg, int T,
                                                int B, int H, int W, int C, int F, float theta, float b_th,
                                                float beta, const int32_t* pool_row_ptr,
                                                const int32_t* pool_col_idx, const float* eps_pool,
                                                int64_t pool_cap, float* dWc, void* workspace,
                                                size_t workspace_bytes, void* stream) {
  if (!trace_in || !V || !arg || !pool_row_ptr || !dWc || !workspace) return SNN_ERR_INVALID_ARG;
  if (pool_cap < 0 || (pool_cap > 0 && (!pool_col_idx || !eps_pool))) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F) || bad_dim(C) || too_big(T, B, H * W * C)) return SNN_ERR_INVALID_ARG;
  if (isnan(theta) || isnan(b_th) || b_th < 0.0f || isnan(beta) || beta < 0.0f) return SNN_ERR_INVALID_ARG;
  if (C * F > 2048) return SNN_ERR_UNSUPPORTED;
  if (workspace_bytes < snn_conv_sparse_dw_workspace(T, B, H, W, C, F)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int TB = T * B;
  const int nb = cdw_blocks(TB, 9 * C * F);
  const int rpb = (TB + nb - 1) / nb;
  const int nacc = 9 * C * F;
  double* part = static_cast<double*>(workspace);
  const size_t lds = (size_t)nacc * sizeof(double);
  const PooledArgs pa{V, arg, theta, b_th, beta};
  auto launch = [&](auto kernel) {
    ensure_dynamic_lds((const void*)kernel, (int)lds);
    hipLaunchKernelGGL(kernel, dim3((unsigned)nb), dim3(kCsdThreads), lds, s, trace_in, TB, H, W, C, F, pool_row_ptr,
                       pool_col_idx, nullptr, eps_pool, pool_cap, rpb, part, pa);
  };
  if (C == 1) launch(conv_dw_sparse_kernel<1, true>);
  else if (C == 2) launch(conv_dw_sparse_kernel<2, true>);
  else launch(conv_dw_sparse_kernel<0, true>);
  hipLaunchKernelGGL(reduce_parts, dim3((unsigned)nacc), dim3(256), 0, s, part, nb, nacc, dWc);
  return launch_status();
}

extern "C" size_t snn_conv_dense_dw_workspace(int T, int B, int H, int W, int C, int F) {
  if (!conv_dims_ok(T, B, H, W, F) || bad_dim(C) || C * F > (1 << 20)) return 0;
  return align256((size_t)dense_blocks((int64_t)T * B * H * W) * 9 * C * F * sizeof(double));
}

extern "C" snn_status snn_conv_dense_dw(const float* trace_in, const float* V, const float* eps_conv, int T, int B,
                                        int H, int W, int C, int F, float theta, float b_th, float beta, float* dWc,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!trace_in || !V || !eps_conv || !dWc || !workspace) return SNN_ERR_INVALID_ARG;
  if (!conv_dims_ok(T, B, H, W, F) || bad_dim(C) || too_big(T, B, H * W * C)) return SNN_ERR_INVALID_ARG;
  if (isnan(theta) || isnan(b_th) || b_th < 0.0f || isnan(beta) || beta < 0.0f) return SNN_ERR_INVALID_ARG;
  if (C * F > (1 << 20)) return SNN_ERR_UNSUPPORTED;
  if (workspace_bytes < snn_conv_dense_dw_workspace(T, B, H, W, C, F)) return SNN_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t n_pos = (int64_t)T * B * H * W;
  const int64_t nb = dense_blocks(n_pos);
  const int64_t ppb = (n_pos + nb - 1) / nb;
  const int nacc = 9 * C * F;
  double* part = static_cast<double*>(workspace);
  if (C == 1)
    hipLaunchKernelGGL(conv_dw_dense_kernel<1>, dim3((unsigned)nb), dim3(kCdwThreads), 0, s, trace_in, V, eps_conv,
                       n_pos, H, W, C, F, theta, b_th, beta, ppb, part);
  else
    hipLaunchKernelGGL(conv_dw_dense_kernel<kDenseMaxC>, dim3((unsigned)nb), dim3(kCdwThreads), 0, s, trace_in, V,
                       eps_conv, n_pos, H, W, C, F, theta, b_th, beta, ppb, part);
  hipLaunchKernelGGL(reduce_parts, dim3((unsigned)nacc), dim3(256), 0, s, part, (int)nb, nacc, dWc);
  return launch_status();
}
