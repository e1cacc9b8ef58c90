// carve_bwd.hip -- the parameter-gradient kernels of the CARVE backward
// (steps 3-6 of the launch sequence in carve_bwd.h), the synchronisation-area
// clear, and the variant dispatch of the fused recompute + adjoint launch.
#include "carve_param.h"

namespace carve {

// The parameter-gradient partials in one launch, one item per workgroup: the
// d[Ub; Uw] items (the heavier ones) first, then the dVb, dVw items, so that
// the second kind fills the compute units the first leaves at its tail.
template <typename T, int D, int RP, bool SW>
__global__ void __launch_bounds__(bwd_threads(D)) carve_bwd_param_kernel(BwdArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int nu = a.B * a.H * kUSplit;
  if ((int)blockIdx.x < nu)
    uparam_item<T, D, RP, SW>(a, blockIdx.x, smem);
  else
    vparam_item<T, D, RP, SW>(a, blockIdx.x - nu, smem);
}

// Sum nparts partial records (2 * half floats each) in a fixed order: thread
// (x, y) of a 64 x 16 block sums records y, y + 16, ... of element x (four
// loads in flight), then the sixteen partial sums are added in order
// y = 0..15.  Elements x < cnt are summed (cnt = 2 * half, or half when there
// is no second half).  blockIdx.y selects the d[Ub; Uw] (0) or the dVb, dVw
// (1) partials, so both reductions share one launch.
constexpr int kReduceGroups = 16;
__global__ void __launch_bounds__(64 * kReduceGroups) carve_param_reduce_kernel(const float* __restrict__ partU,
                                                                                int npartU,
                                                                                const float* __restrict__ partV,
                                                                                int npartV, size_t half, size_t cnt,
                                                                                float* dU0, float* dU1, float* dV0,
                                                                                float* dV1) {
  const float* part = blockIdx.y == 0 ? partU : partV;
  const int nparts = blockIdx.y == 0 ? npartU : npartV;
  float* dst0 = blockIdx.y == 0 ? dU0 : dV0;
  float* dst1 = blockIdx.y == 0 ? dU1 : dV1;
  __shared__ float red[kReduceGroups][64];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const size_t x = (size_t)blockIdx.x * 64 + tx;
  const size_t n = 2 * half;
  float s = 0.0f;
  if (x < cnt) {
    const float* p = part + x;
    constexpr int G = kReduceGroups;
    int q = ty;
    for (; q + 3 * G < nparts; q += 4 * G) {
      const float a0 = p[(size_t)q * n], a1 = p[(size_t)(q + G) * n];
      const float a2 = p[(size_t)(q + 2 * G) * n], a3 = p[(size_t)(q + 3 * G) * n];
      s += a0;
      s += a1;
      s += a2;
      s += a3;
    }
    for (; q < nparts; q += G) s += p[(size_t)q * n];
  }
  red[ty][tx] = s;
  __syncthreads();
  if (ty == 0 && x < cnt) {
    float t = red[0][tx];
    for (int y = 1; y < kReduceGroups; ++y) t += red[y][tx];
    if (x < half) dst0[x] = t;
    else dst1[x - half] = t;
  }
}

// Reverse mode of the query / key activation (kVarAct), in place: with
// s = SiLU(raw) over a row of D channels, n = sqrt(|s|^2 + eps) and y = s / n,
//   d raw = (dy - y (y . dy)) / n * SiLU'(raw).
// One 16-byte chunk per thread; a row's D / VEC chunks are consecutive threads
// of one wave, so the two row sums run over those lanes.  blockIdx.y selects
// q (0) or k (1).
template <typename T, int D>
__global__ void __launch_bounds__(256) carve_act_bwd_kernel(const T* __restrict__ qraw, const T* __restrict__ kraw,
                                                            T* __restrict__ dq, T* __restrict__ dk, size_t rows) {
  constexpr int VEC = 16 / sizeof(T), NC = D / VEC, N = Chunk16<T>::N;
  static_assert(256 % NC == 0 && NC <= 64, "rows inside one wave");
  const T* raw = blockIdx.y ? kraw : qraw;
  T* dy = blockIdx.y ? dk : dq;
  const size_t n = rows * NC;
  const size_t x = (size_t)blockIdx.x * 256 + threadIdx.x;
  // a row is wholly inside or outside [0, n): lanes past the end work on the
  // last chunk (every lane takes part in the row sums) and store nothing
  const size_t xc = x < n ? x : n - 1;
  float f[N], d[N], sv[N];
  Chunk16<T>::unpack(*reinterpret_cast<const u32x4_t*>(raw + xc * VEC), f);
  Chunk16<T>::unpack(*reinterpret_cast<const u32x4_t*>(dy + xc * VEC), d);
  float ss = 0.0f;
  for (int i = 0; i < N; ++i) {
    sv[i] = silu_f(f[i]);
    ss += sv[i] * sv[i];
  }
  const float inv = rsqrtf(group_sum<NC>(ss) + kL2Eps);
  float dot = 0.0f;
  for (int i = 0; i < N; ++i) dot += sv[i] * inv * d[i];
  dot = group_sum<NC>(dot);
  for (int i = 0; i < N; ++i) d[i] = (d[i] - sv[i] * inv * dot) * inv * silu_grad_f(f[i]);
  if (x < n) *reinterpret_cast<u32x4_t*>(dy + x * VEC) = Chunk16<T>::pack(d);
}

template <typename T, int D>
static int launch_act_bwd_t(const void* qr, const void* kr, void* dq, void* dk, size_t rows, hipStream_t s) {
  constexpr int NC = D / (16 / sizeof(T));
  const size_t blocks = (rows * NC + 255) / 256;
  hipLaunchKernelGGL((carve_act_bwd_kernel<T, D>), dim3((unsigned)blocks, 2), dim3(256), 0, s,
                     reinterpret_cast<const T*>(qr), reinterpret_cast<const T*>(kr), reinterpret_cast<T*>(dq),
                     reinterpret_cast<T*>(dk), rows);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T>
static int launch_act_bwd_d(const void* qr, const void* kr, void* dq, void* dk, size_t rows, int D, hipStream_t s) {
  if (D == 32) return launch_act_bwd_t<T, 32>(qr, kr, dq, dk, rows, s);
  if (D == 64) return launch_act_bwd_t<T, 64>(qr, kr, dq, dk, rows, s);
  if (D == 128) return launch_act_bwd_t<T, 128>(qr, kr, dq, dk, rows, s);
  return CARVE_ERR_UNSUPPORTED;
}

int launch_act_bwd(const void* q_raw, const void* k_raw, void* dq, void* dk, size_t rows, int D, int dtype,
                   hipStream_t s) {
  if (rows == 0) return CARVE_OK;
  if (dtype == CARVE_BF16) return launch_act_bwd_d<bf16_t>(q_raw, k_raw, dq, dk, rows, D, s);
  return launch_act_bwd_d<float>(q_raw, k_raw, dq, dk, rows, D, s);
}

// Zero the synchronisation area of the fused launch (ready flags, ticket).
__global__ void __launch_bounds__(256) carve_sync_clear_kernel(int* __restrict__ sync, int n) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x < n) sync[x] = 0;
}

int launch_sync_clear(int* sync, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(carve_sync_clear_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, sync, (int)n);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

int launch_bwd_fused(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int dtype, int D, int LW,
                     int var, hipStream_t s) {
  switch (var) {
    case 0: return launch_bwd_fused_var<0>(f, a, sync, cus, dtype, D, LW, s);
    case kVarGated: return launch_bwd_fused_var<kVarGated>(f, a, sync, cus, dtype, D, LW, s);
    case kVarScalarW: return launch_bwd_fused_var<kVarScalarW>(f, a, sync, cus, dtype, D, LW, s);
    case kVarGated | kVarScalarW:
      return launch_bwd_fused_var<kVarGated | kVarScalarW>(f, a, sync, cus, dtype, D, LW, s);
    case kVarAct: return launch_bwd_fused_var<kVarAct>(f, a, sync, cus, dtype, D, LW, s);
    default: return CARVE_ERR_UNSUPPORTED;
  }
}

// dA[h][j] and dtau[h][j] as sums over b = 0, 1, ... (in order) of the
// per-(batch, head) partials (layout [B*H][2][D]); one thread per (h, j)
__global__ void __launch_bounds__(256) carve_gate_reduce_kernel(const float* __restrict__ partG, int B, int H, int D,
                                                                float* __restrict__ dA, float* __restrict__ dtau) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x >= H * D) return;
  const int h = x / D, j = x % D;
  float sa = 0.0f, st = 0.0f;
  for (int b = 0; b < B; ++b) {
    const float* p = partG + ((size_t)b * H + h) * 2 * D;
    sa += p[j];
    st += p[D + j];
  }
  dA[x] = sa;
  dtau[x] = st;
}

int launch_gate_reduce(const float* partG, int B, int H, int D, float* dA, float* dtau, hipStream_t s) {
  hipLaunchKernelGGL(carve_gate_reduce_kernel, dim3((unsigned)((H * D + 255) / 256)), dim3(256), 0, s, partG, B, H, D,
                     dA, dtau);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T, int D, int RP>
static size_t fused_lds_l(int LW) {
  if (LW == 16) return fused_lds<T, D, 16, RP, 0>();
  if (LW == 32) return fused_lds<T, D, 32, RP, 0>();
  return (size_t)-1;
}

template <typename T>
static size_t fused_lds_d(int D, int LW, int RP) {
  if (RP == 32) {
    if (D == 32) return fused_lds_l<T, 32, 32>(LW);
    if (D == 64) return fused_lds_l<T, 64, 32>(LW);
    if (D == 128) return fused_lds_l<T, 128, 32>(LW);
  } else if (RP == 64) {
    if (D == 32) return fused_lds_l<T, 32, 64>(LW);
    if (D == 64) return fused_lds_l<T, 64, 64>(LW);
    if (D == 128) return fused_lds_l<T, 128, 64>(LW);
  }
  return (size_t)-1;
}

size_t bwd_lds_bytes(int dtype, int D, int LW, int RP) {
  return dtype == CARVE_BF16 ? fused_lds_d<bf16_t>(D, LW, RP) : fused_lds_d<float>(D, LW, RP);
}

template <typename T, int D, int RP, bool SW>
static int launch_param_s(const BwdArgs& a, hipStream_t s) {
  constexpr size_t lu = uparam_lds<T, D, SW ? RP : 2 * RP>(), lv = vparam_lds<T, D, RP, SW>();
  constexpr size_t lds = lu > lv ? lu : lv;
  if constexpr (lds > 64 * 1024) {
    return CARVE_ERR_UNSUPPORTED;   // only shapes the fused launch rejects first
  } else {
    hipLaunchKernelGGL((carve_bwd_param_kernel<T, D, RP, SW>), dim3(a.B * a.H * (kUSplit + kVSplit)),
                       dim3(bwd_threads(D)), lds, s, a);
    return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
  }
}

template <typename T, int D, int RP>
static int launch_param_t(const BwdArgs& a, bool sw, hipStream_t s) {
  return sw ? launch_param_s<T, D, RP, true>(a, s) : launch_param_s<T, D, RP, false>(a, s);
}

template <typename T>
static int launch_param_d(const BwdArgs& a, int D, bool sw, hipStream_t s) {
  if (a.RP == 32) {
    if (D == 32) return launch_param_t<T, 32, 32>(a, sw, s);
    if (D == 64) return launch_param_t<T, 64, 32>(a, sw, s);
    if (D == 128) return launch_param_t<T, 128, 32>(a, sw, s);
  } else if (a.RP == 64) {
    if (D == 32) return launch_param_t<T, 32, 64>(a, sw, s);
    if (D == 64) return launch_param_t<T, 64, 64>(a, sw, s);
    if (D == 128) return launch_param_t<T, 128, 64>(a, sw, s);
  }
  return CARVE_ERR_UNSUPPORTED;
}

int launch_bwd_param(const BwdArgs& a, int dtype, int D, bool sw, hipStream_t s) {
  if (dtype == CARVE_BF16) return launch_param_d<bf16_t>(a, D, sw, s);
  return launch_param_d<float>(a, D, sw, s);
}

int launch_param_reduce(const float* partU, int npartU, const float* partV, int npartV, size_t half, float* dU0,
                        float* dU1, float* dV0, float* dV1, hipStream_t s) {
  const size_t cnt = dU1 ? 2 * half : half;
  const int blocks = (int)((cnt + 63) / 64);
  hipLaunchKernelGGL(carve_param_reduce_kernel, dim3(blocks, 2), dim3(64 * kReduceGroups), 0, s, partU, npartU, partV,
                     npartV, half, cnt, dU0, dU1, dV0, dV1);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

}  // namespace carve
