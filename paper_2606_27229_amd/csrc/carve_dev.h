// carve_dev.h -- device-side building blocks shared by the CARVE kernels
// (gfx950 / CDNA4, wave64).
//
// Matrix-core tiles.  Every product in the layer is issued as 16x16 output
// tiles on the MFMA units:
//   bf16 operands: v_mfma_f32_16x16x32_bf16 (8 bf16 of K per lane)
//   f32  operands: v_mfma_f32_16x16x4_f32   (1 f32 of K per lane)
// Operand fragments: lane l = 16*g + c supplies row (c) of A / column (c) of B
// and the K-slots [g*KPL, (g+1)*KPL).  The f32 result of a tile lives in four
// registers per lane: rows 4g+r (r = 0..3) of column c.  Both operands are read
// K-contiguously ("A row-major [m][k]", "B stored as [n][k]"), so every LDS
// operand buffer below is laid out with its contraction index innermost.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace carve {

template <typename T>
struct Mma;

template <>
struct Mma<bf16_t> {
  static constexpr int KS = 32;   // K per instruction
  static constexpr int KPL = 8;   // K values per lane
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const bf16_t* p) {
    return *reinterpret_cast<const bf16x8*>(p);
  }
  static __device__ __forceinline__ frag load_scaled(const bf16_t* p, const float* s) {
    bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
    const f32x4 s0 = *reinterpret_cast<const f32x4*>(s);
    const f32x4 s1 = *reinterpret_cast<const f32x4*>(s + 4);
    bf16x8 o;
    o[0] = (bf16_t)((float)v[0] * s0[0]);
    o[1] = (bf16_t)((float)v[1] * s0[1]);
    o[2] = (bf16_t)((float)v[2] * s0[2]);
    o[3] = (bf16_t)((float)v[3] * s0[3]);
    o[4] = (bf16_t)((float)v[4] * s1[0]);
    o[5] = (bf16_t)((float)v[5] * s1[1]);
    o[6] = (bf16_t)((float)v[6] * s1[2]);
    o[7] = (bf16_t)((float)v[7] * s1[3]);
    return o;
  }
  // fragment built from f32 values (8 consecutive)
  static __device__ __forceinline__ frag from_f32(const float* p) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
    bf16x8 o;
    o[0] = (bf16_t)a[0]; o[1] = (bf16_t)a[1]; o[2] = (bf16_t)a[2]; o[3] = (bf16_t)a[3];
    o[4] = (bf16_t)b[0]; o[5] = (bf16_t)b[1]; o[6] = (bf16_t)b[2]; o[7] = (bf16_t)b[3];
    return o;
  }
  static __device__ __forceinline__ frag zero() {
    bf16x8 o;
    for (int e = 0; e < 8; ++e) o[e] = (bf16_t)0.0f;
    return o;
  }
};

template <>
struct Mma<float> {
  static constexpr int KS = 4;
  static constexpr int KPL = 1;
  typedef float frag;
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
  static __device__ __forceinline__ frag load_scaled(const float* p, const float* s) {
    return p[0] * s[0];
  }
  static __device__ __forceinline__ frag from_f32(const float* p) { return *p; }
  static __device__ __forceinline__ frag zero() { return 0.0f; }
};

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

template <typename T>
__device__ __forceinline__ T to_t(float x) { return (T)x; }

template <typename T>
__device__ __forceinline__ float to_f(T x) { return (float)x; }

// ---- result-tile stores ----------------------------------------------------
// Tile (rows r0.., cols c0..) of the C layout into a row-major buffer.
template <typename T>
__device__ __forceinline__ void store_tile(T* buf, int ld, int r0, int c0, f32x4 v, int lane) {
  const int g = lane >> 4, c = lane & 15;
  T* p = buf + (size_t)(r0 + 4 * g) * ld + c0 + c;
  p[0] = (T)v[0];
  p[ld] = (T)v[1];
  p[2 * ld] = (T)v[2];
  p[3 * ld] = (T)v[3];
}

// Tile stored transposed: element (row, col) goes to buf[col * ld + row]; the
// four rows a lane holds are contiguous.
__device__ __forceinline__ void store_tile_t(bf16_t* buf, int ld, int r0, int c0, f32x4 v, int lane) {
  const int g = lane >> 4, c = lane & 15;
  bf16x4 o;
  o[0] = (bf16_t)v[0]; o[1] = (bf16_t)v[1]; o[2] = (bf16_t)v[2]; o[3] = (bf16_t)v[3];
  *reinterpret_cast<bf16x4*>(buf + (size_t)(c0 + c) * ld + r0 + 4 * g) = o;
}
__device__ __forceinline__ void store_tile_t(float* buf, int ld, int r0, int c0, f32x4 v, int lane) {
  const int g = lane >> 4, c = lane & 15;
  *reinterpret_cast<f32x4*>(buf + (size_t)(c0 + c) * ld + r0 + 4 * g) = v;
}

// ---- elementwise math (f32, hardware exp2/log2/rcp) -----------------------
__device__ __forceinline__ float fast_exp(float x) { return __expf(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float sigmoid_f(float z) { return fast_rcp(1.0f + fast_exp(-z)); }
// log(1 + e^z) without overflow
__device__ __forceinline__ float softplus_f(float z) {
  return fmaxf(z, 0.0f) + __logf(1.0f + fast_exp(-fabsf(z)));
}
// tanh with a short odd series near 0 (the exp form cancels there)
__device__ __forceinline__ float tanh_f(float y) {
  const float big = 1.0f - 2.0f * fast_rcp(fast_exp(2.0f * y) + 1.0f);
  const float y2 = y * y;
  const float small = y * (1.0f + y2 * (-1.0f / 3.0f + y2 * (2.0f / 15.0f + y2 * (-17.0f / 315.0f))));
  return fabsf(y) < 0.125f ? small : big;
}

}  // namespace carve
