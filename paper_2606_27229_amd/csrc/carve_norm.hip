// carve_norm.hip -- the output RMS normalisation of the layer: the step that
// closes Alg. carve_fwd, y = W_O RMSNorm(reshape(o)), without W_O (a plain
// GEMM outside the recurrence).  The paper runs it as one hoisted launch over
// the assembled o (Alg. megakernel) and its gradient as the mirrored hoisted
// launch of Alg. megakernel_bwd; so do these row kernels.
//
// A token's row is reshape(o)[b, t, :], the N = H * Dv values of all its heads
// ([B, T, H, Dv] row-major is [B*T, N] row-major):
//   r = 1 / sqrt(mean_i x_i^2 + eps),  n = x r,  y = n * weight
// and for loss <dy, y>:
//   dn = dy * weight,  dx = r (dn - n mean_i(dn_i n_i)),  dweight = sum_rows dy * n
//
// One wave per row.  Lane l holds the 16-byte chunks l, l + 64, ... of the row
// (NCH of them), so every load and store of a wave covers 1 KB of contiguous
// row; the row sums are butterfly reductions over the wave.  The backward runs
// a fixed grid: wave x of the grid takes rows x, x + (waves in the grid), ...
// and keeps its share of dweight in registers; the workgroup sums its waves in
// order into one partial row, and a second kernel sums the partials in order,
// so reruns are bitwise identical.
#include <mutex>

#include "carve_kernels.h"

// Scratch of carve_rmsnorm_bwd_noalloc, for callers that cannot allocate: the
// dweight partial rows of the backward (at most kNormBwdGroups rows of at most
// 4096 floats).  Each GPU the library runs on holds its own copy until the
// process ends.  Host code never uses this name as an address: the device
// address comes from hipGetSymbolAddress, once per device (norm_scratch).
static __device__ __align__(256) float scratch[carve::kNormScratchBytes / sizeof(float)];

namespace carve {

namespace {

constexpr int kNormWaves = 4;   // waves (rows in flight) per workgroup

template <typename T>
struct NormVec;
template <>
struct NormVec<bf16_t> {
  static constexpr int n = 8;
  typedef bf16x8 v;
};
template <>
struct NormVec<float> {
  static constexpr int n = 4;
  typedef f32x4 v;
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

template <typename T, int NCH>
__global__ void __launch_bounds__(64 * kNormWaves)
    carve_rmsnorm_fwd_kernel(const T* __restrict__ x, const float* __restrict__ wt, T* __restrict__ y, long rows,
                             int N, float eps) {
  typedef typename NormVec<T>::v vec;
  constexpr int VEC = NormVec<T>::n;
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * kNormWaves + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* xr = x + row * N;
  vec xv[NCH];
  float ss = 0.0f;
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int c0 = (ch * 64 + lane) * VEC;
    if (c0 < N) {
      xv[ch] = *reinterpret_cast<const vec*>(xr + c0);
#pragma unroll
      for (int e = 0; e < VEC; ++e) ss += (float)xv[ch][e] * (float)xv[ch][e];
    }
  }
  const float r = 1.0f / sqrtf(wave_sum(ss) / (float)N + eps);
  T* yr = y + row * N;
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int c0 = (ch * 64 + lane) * VEC;
    if (c0 < N) {
      vec o;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[e] = (T)((float)xv[ch][e] * r * wt[c0 + e]);
      *reinterpret_cast<vec*>(yr + c0) = o;
    }
  }
}

// grid: nwg workgroups; partial[blockIdx.x][N] f32 receives the workgroup's
// dweight share (its waves summed in order)
template <typename T, int NCH>
__global__ void __launch_bounds__(64 * kNormWaves)
    carve_rmsnorm_bwd_kernel(const T* __restrict__ x, const float* __restrict__ wt, const T* __restrict__ dy,
                             T* __restrict__ dx, float* __restrict__ partial, long rows, int N, float eps) {
  typedef typename NormVec<T>::v vec;
  constexpr int VEC = NormVec<T>::n;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* sacc = reinterpret_cast<float*>(smem);   // [kNormWaves][N]
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long stride = (long)gridDim.x * kNormWaves;
  float acc[NCH][VEC];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[ch][e] = 0.0f;
  for (long row = (long)blockIdx.x * kNormWaves + wv; row < rows; row += stride) {
    const T* xr = x + row * N;
    const T* dyr = dy + row * N;
    vec xv[NCH], dv[NCH];
    float ss = 0.0f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int c0 = (ch * 64 + lane) * VEC;
      if (c0 < N) {
        xv[ch] = *reinterpret_cast<const vec*>(xr + c0);
        dv[ch] = *reinterpret_cast<const vec*>(dyr + c0);
#pragma unroll
        for (int e = 0; e < VEC; ++e) ss += (float)xv[ch][e] * (float)xv[ch][e];
      }
    }
    const float r = 1.0f / sqrtf(wave_sum(ss) / (float)N + eps);
    float dot = 0.0f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int c0 = (ch * 64 + lane) * VEC;
      if (c0 < N) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float n = (float)xv[ch][e] * r, d = (float)dv[ch][e];
          dot += d * wt[c0 + e] * n;
          acc[ch][e] += d * n;
        }
      }
    }
    const float m = wave_sum(dot) / (float)N;
    T* dxr = dx + row * N;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int c0 = (ch * 64 + lane) * VEC;
      if (c0 < N) {
        vec o;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float n = (float)xv[ch][e] * r;
          o[e] = (T)(r * ((float)dv[ch][e] * wt[c0 + e] - n * m));
        }
        *reinterpret_cast<vec*>(dxr + c0) = o;
      }
    }
  }
  // the workgroup's partial: its waves' shares summed in wave order
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int c0 = (ch * 64 + lane) * VEC;
    if (c0 < N)
#pragma unroll
      for (int e = 0; e < VEC; ++e) sacc[wv * N + c0 + e] = acc[ch][e];
  }
  __syncthreads();
  for (int col = threadIdx.x; col < N; col += 64 * kNormWaves) {
    float s = 0.0f;
    for (int w = 0; w < kNormWaves; ++w) s += sacc[w * N + col];
    partial[(size_t)blockIdx.x * N + col] = s;
  }
}

// dweight[col] = the sum of partial[g][col] over g in a fixed order: thread
// (x, y) of a 64 x 16 block sums partials y, y + 16, ... of column x (four
// loads in flight), then the sixteen sums are added in order y = 0..15
constexpr int kNormReduceGroups = 16;
__global__ void __launch_bounds__(64 * kNormReduceGroups)
    carve_rmsnorm_reduce_kernel(const float* __restrict__ partial, int nparts, int N, float* __restrict__ dw) {
  __shared__ float red[kNormReduceGroups][64];
  constexpr int G = kNormReduceGroups;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + tx;
  float s = 0.0f;
  if (col < N) {
    const float* p = partial + col;
    int g = ty;
    for (; g + 3 * G < nparts; g += 4 * G) {
      const float a0 = p[(size_t)g * N], a1 = p[(size_t)(g + G) * N];
      const float a2 = p[(size_t)(g + 2 * G) * N], a3 = p[(size_t)(g + 3 * G) * N];
      s += a0;
      s += a1;
      s += a2;
      s += a3;
    }
    for (; g < nparts; g += G) s += p[(size_t)g * N];
  }
  red[ty][tx] = s;
  __syncthreads();
  if (ty == 0 && col < N) {
    float t = red[0][tx];
    for (int y = 1; y < G; ++y) t += red[y][tx];
    dw[col] = t;
  }
}

template <typename T>
int nch_of(int N) {
  for (int nch = 1; nch <= 8; nch *= 2)
    if (N <= 64 * nch * NormVec<T>::n) return nch;
  return 0;
}

template <typename T, int NCH>
int launch_fwd_t(const void* x, const float* wt, void* y, long rows, int N, float eps, hipStream_t s) {
  const long nwg = (rows + kNormWaves - 1) / kNormWaves;
  hipLaunchKernelGGL((carve_rmsnorm_fwd_kernel<T, NCH>), dim3((unsigned)nwg), dim3(64 * kNormWaves), 0, s,
                     reinterpret_cast<const T*>(x), wt, reinterpret_cast<T*>(y), rows, N, eps);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T, int NCH>
int launch_bwd_t(const void* x, const float* wt, const void* dy, void* dx, float* partial, int nwg, long rows, int N,
                 float eps, hipStream_t s) {
  const size_t lds = (size_t)kNormWaves * N * sizeof(float);
  hipLaunchKernelGGL((carve_rmsnorm_bwd_kernel<T, NCH>), dim3((unsigned)nwg), dim3(64 * kNormWaves), lds, s,
                     reinterpret_cast<const T*>(x), wt, reinterpret_cast<const T*>(dy), reinterpret_cast<T*>(dx),
                     partial, rows, N, eps);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T>
int launch_fwd_d(const void* x, const float* wt, void* y, long rows, int N, float eps, hipStream_t s) {
  switch (nch_of<T>(N)) {
    case 1: return launch_fwd_t<T, 1>(x, wt, y, rows, N, eps, s);
    case 2: return launch_fwd_t<T, 2>(x, wt, y, rows, N, eps, s);
    case 4: return launch_fwd_t<T, 4>(x, wt, y, rows, N, eps, s);
    case 8: return launch_fwd_t<T, 8>(x, wt, y, rows, N, eps, s);
    default: return CARVE_ERR_UNSUPPORTED;
  }
}

template <typename T>
int launch_bwd_d(const void* x, const float* wt, const void* dy, void* dx, float* partial, int nwg, long rows, int N,
                 float eps, hipStream_t s) {
  switch (nch_of<T>(N)) {
    case 1: return launch_bwd_t<T, 1>(x, wt, dy, dx, partial, nwg, rows, N, eps, s);
    case 2: return launch_bwd_t<T, 2>(x, wt, dy, dx, partial, nwg, rows, N, eps, s);
    case 4: return launch_bwd_t<T, 4>(x, wt, dy, dx, partial, nwg, rows, N, eps, s);
    case 8: return launch_bwd_t<T, 8>(x, wt, dy, dx, partial, nwg, rows, N, eps, s);
    default: return CARVE_ERR_UNSUPPORTED;
  }
}

}  // namespace

bool rmsnorm_supported(int dtype, int N) {
  if (dtype == CARVE_BF16) return N % NormVec<bf16_t>::n == 0 && nch_of<bf16_t>(N) != 0;
  return N % NormVec<float>::n == 0 && nch_of<float>(N) != 0;
}

int rmsnorm_bwd_groups(long rows) {
  const long nwg = (rows + kNormWaves - 1) / kNormWaves;
  return (int)(nwg < kNormBwdGroups ? nwg : kNormBwdGroups);
}

int launch_rmsnorm_fwd(const void* x, const float* wt, void* y, long rows, int N, float eps, int dtype,
                       hipStream_t s) {
  if (dtype == CARVE_BF16) return launch_fwd_d<bf16_t>(x, wt, y, rows, N, eps, s);
  return launch_fwd_d<float>(x, wt, y, rows, N, eps, s);
}

int launch_rmsnorm_bwd(const void* x, const float* wt, const void* dy, void* dx, float* partial, float* dw, long rows,
                       int N, float eps, int dtype, hipStream_t s, void (*mark)(hipStream_t)) {
  const int nwg = rmsnorm_bwd_groups(rows);
  const int st = dtype == CARVE_BF16 ? launch_bwd_d<bf16_t>(x, wt, dy, dx, partial, nwg, rows, N, eps, s)
                                     : launch_bwd_d<float>(x, wt, dy, dx, partial, nwg, rows, N, eps, s);
  if (st) return st;
  if (mark) mark(s);
  hipLaunchKernelGGL(carve_rmsnorm_reduce_kernel, dim3((unsigned)((N + 63) / 64)), dim3(64 * kNormReduceGroups), 0, s,
                     partial, nwg, N, dw);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

}  // namespace carve

namespace carve {

// The device address of this device's scratch array (looked up on the first
// call made with the device current, then cached), or CARVE_ERR_HIP.
int norm_scratch(float** ptr) {
  static std::mutex mu;
  static float* addr[kMaxNormDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxNormDevices) return CARVE_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CARVE_ERR_HIP;
    addr[dev] = reinterpret_cast<float*>(p);
  }
  *ptr = addr[dev];
  return CARVE_OK;
}

}  // namespace carve
