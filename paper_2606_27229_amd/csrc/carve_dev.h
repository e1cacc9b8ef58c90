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

// ---- K16 "quad" operands --------------------------------------------------
// The kernels issue their products on K16 (and paired K32) matrix-core steps.
// For one 16x16 output tile and one 16-wide slice of the contraction index k:
//   lane l = 16 g + c supplies A[m = c][k = 4g .. 4g+3]  and  B[k = 4g .. 4g+3][n = c]
//   and receives C[m = 4g + i][n = c], i = 0..3.
// So an accumulator tile X held in registers is directly a B operand whose K is
// X's row index, and an A operand representing X^T.  LDS operands are read as
// 4-element quads either along a row ("natural": lane c reads row c) or across
// four rows ("transposed": lane c reads column c), the latter with the gfx950
// transposing LDS read for 16-bit data.
template <typename T>
struct Quad;

template <>
struct Quad<bf16_t> {
  typedef bf16x4 q;
  static __device__ __forceinline__ q ld(const bf16_t* p) { return *reinterpret_cast<const bf16x4*>(p); }
  // lane (g, c) receives buf[r0 + 4g + e][c0 + c], e = 0..3
  static __device__ __forceinline__ q ld_tr(const bf16_t* buf, int ld, int r0, int c0, int g, int c) {
    typedef short short4_ __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) short4_ lds_s4;
    const bf16_t* p = buf + (r0 + 4 * g + (c >> 2)) * ld + c0 + 4 * (c & 3);
    const short4_ v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p));
    return __builtin_bit_cast(bf16x4, v);
  }
  // ld_tr on a quad-swizzled tile (qswz below); r0 a multiple of 16, so the
  // swizzle term of every row this lane touches is g
  static __device__ __forceinline__ q ld_tr_sw(const bf16_t* buf, int ld, int r0, int c0, int g, int c) {
    return ld_tr_at(buf + (r0 + 4 * g + (c >> 2)) * ld + c0 + 4 * ((c & 3) ^ g));
  }
  // transposing read with the lane's own address (lane (g, c) names row
  // r0 + 4 g + c / 4, quad c % 4 of the 16 columns)
  static __device__ __forceinline__ q ld_tr_at(const bf16_t* p) {
    typedef short short4_ __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) short4_ lds_s4;
    const short4_ v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p));
    return __builtin_bit_cast(bf16x4, v);
  }
  static __device__ __forceinline__ void st(bf16_t* p, q v) { *reinterpret_cast<bf16x4*>(p) = v; }
  static __device__ __forceinline__ q cvt(f32x4 x) {
    q o;
    o[0] = (bf16_t)x[0]; o[1] = (bf16_t)x[1]; o[2] = (bf16_t)x[2]; o[3] = (bf16_t)x[3];
    return o;
  }
  static __device__ __forceinline__ f32x4 f32(q x) {
    f32x4 o = {(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
    return o;
  }
  static __device__ __forceinline__ f32x4 mma16(q a, q b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
  }
  // two K16 slices in one K32 step (the same slice pairing on both sides)
  static __device__ __forceinline__ f32x4 mma32(q a0, q a1, q b0, q b1, f32x4 c) {
    const bf16x8 a = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
    const bf16x8 b = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Quad<float> {
  typedef f32x4 q;
  static __device__ __forceinline__ q ld(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  static __device__ __forceinline__ q ld_tr(const float* buf, int ld, int r0, int c0, int g, int c) {
    const float* p = buf + (r0 + 4 * g) * ld + c0 + c;
    q o = {p[0], p[ld], p[2 * ld], p[3 * ld]};
    return o;
  }
  // f32 tiles are not swizzled (qswz<float> is 0)
  static __device__ __forceinline__ q ld_tr_sw(const float* buf, int ld, int r0, int c0, int g, int c) {
    return ld_tr(buf, ld, r0, c0, g, c);
  }
  static __device__ __forceinline__ void st(float* p, q v) { *reinterpret_cast<f32x4*>(p) = v; }
  static __device__ __forceinline__ q cvt(f32x4 x) { return x; }
  static __device__ __forceinline__ f32x4 f32(q x) { return x; }
  static __device__ __forceinline__ f32x4 mma16(q a, q b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ f32x4 mma32(q a0, q a1, q b0, q b1, f32x4 c) {
    return mma16(a1, b1, mma16(a0, b0, c));
  }
};

// ---- bank-conflict-free bf16 operand tiles -----------------------------------
// The LDS serves 8-byte lane accesses in groups: reads (row-wise or
// transposing) 32 lanes at a time against a 256-byte bank window, writes 16
// lanes at a time against a 128-byte window.  A row-major bf16 tile is read and
// written in three quad (8-byte) patterns: 16 rows x 2 quads (row-wise read),
// 8 rows x 4 quads (transposing read) and 16 rows x 1 quad (write of a result
// tile).  Row padding alone cannot make all three conflict-free.  With a row
// stride of x quads, x = 4 (mod 8), and quad q of row r stored at quad
// q ^ ((r >> 2) & 3), all three are: the XOR spreads the rows that the stride
// maps to one window position.  The term only touches the quad index's two low
// bits, so offsets along a row stay additive.
// qswz<T>(r): the element-index XOR of row r (f32 tiles: none).
template <typename T>
__device__ __forceinline__ int qswz(int r) {
  return sizeof(T) == 2 ? ((r >> 2) & 3) << 2 : 0;
}
// The same three patterns on unpadded 256-byte bf16 rows (128 elements, 32
// quads): quad q of row r at quad q ^ hq(r mod 16), hq linear over the bits of
// r with images 4, 8, 17, 2.  hq mod 16 is a bijection of the 16 rows (writes),
// and {1, 2, 4, 8, 17} is a basis of the quad index (both reads).
// hswz128(r): the element-index XOR of row r.
__device__ __forceinline__ int hswz128(int r) {
  return (((r & 1) ? 4 : 0) ^ ((r & 2) ? 8 : 0) ^ ((r & 4) ? 17 : 0) ^ ((r & 8) ? 2 : 0)) << 2;
}
// Transposing read (rows r0 + 4 g + c / 4, columns c0 + 4 (c % 4), r0 a
// multiple of 16) of a tile laid out with hswz128 (SXH: rows of LD = 128
// elements; sxo = the lane's offset of row 4 g + c / 4 with its swizzle term,
// computed once), or of a plain padded tile.
template <bool SXH, typename T, int LD>
__device__ __forceinline__ typename Quad<T>::q ld_sx_tile(const T* buf, int r0, int sxo, int c0, int g, int c) {
  if constexpr (SXH) return Quad<T>::ld_tr_at(buf + r0 * LD + sxo);
  else return Quad<T>::ld_tr(buf, LD, r0, c0, g, c);
}
// sxo of ld_sx_tile for the column block c0
__device__ __forceinline__ int sx_lane_offset(int c0, int g, int c) {
  const int r = 4 * g + (c >> 2);
  return r * 128 + ((c0 + 4 * (c & 3)) ^ hswz128(r));
}

// global 4-element vector of the token dtype <-> f32x4
__device__ __forceinline__ f32x4 gload4(const bf16_t* p) {
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  f32x4 o = {(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
  return o;
}
__device__ __forceinline__ f32x4 gload4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// DPP helpers inside rows of 16 lanes
// x of the lane one to the left in its row; the first lane of a row gets fill
__device__ __forceinline__ float row_shr1(float x, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill), __builtin_bit_cast(int, x),
                                                               0x111, 0xf, 0xf, false));
}
// x of the lane one to the right in its row; the last lane of a row gets fill
__device__ __forceinline__ float row_shl1(float x, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill), __builtin_bit_cast(int, x),
                                                               0x101, 0xf, 0xf, false));
}
// x of lane 15 of the row, in every lane of the row (every lane is written, so
// no old value is needed)
__device__ __forceinline__ float row_bcast15(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x15F, 0xf, 0xf, false));
}
// x of the neighbouring lane (lane ^ 1)
__device__ __forceinline__ float lane_xor1(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xf, 0xf, false));
}
// wait until every vector memory operation this wave issued has completed
__device__ __forceinline__ void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// inclusive suffix sum over the 16 lanes of each row
__device__ __forceinline__ float row_suffix(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x101, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x102, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x104, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x108, 0xf, 0xf, false));
  return x;
}
// inclusive prefix sum over the 16 lanes of each row
__device__ __forceinline__ float row_scan(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x111, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x112, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x114, 0xf, 0xf, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x118, 0xf, 0xf, false));
  return x;
}

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
// base-2 forms for code that keeps log retentions in units of log 2 (every
// exponential then is one hardware exp2, with no scaling product)
constexpr float kLog2e = 1.44269504088896341f;
__device__ __forceinline__ float exp2_f(float y) { return __builtin_amdgcn_exp2f(y); }
// 2^y and 2^-y
__device__ __forceinline__ void exp2_pm(float y, float& ep, float& em) {
  ep = __builtin_amdgcn_exp2f(y);
  em = __builtin_amdgcn_exp2f(-y);
}
// softplus(z) / log 2 = log2(1 + e^z) without overflow (the log2 argument is
// in [1, 2])
__device__ __forceinline__ float softplus2_f(float z) {
  return fmaf(fmaxf(z, 0.0f), kLog2e, __builtin_amdgcn_logf(1.0f + __builtin_amdgcn_exp2f(-fabsf(z) * kLog2e)));
}
// natural log of x in [1, 2]: the hardware log2 and one product (no range
// reduction or denormal scaling is needed there)
__device__ __forceinline__ float log_1to2(float x) { return __builtin_amdgcn_logf(x) * 0.693147180559945f; }
// log(1 + e^z) without overflow
__device__ __forceinline__ float softplus_f(float z) {
  return fmaxf(z, 0.0f) + log_1to2(1.0f + fast_exp(-fabsf(z)));
}
// softplus(z) = log(1 + e^z) and sigmoid(z) from one exponential
__device__ __forceinline__ void softplus_sigmoid(float z, float& sp, float& sig) {
  const float e = fast_exp(-fabsf(z));
  const float r = fast_rcp(1.0f + e);
  sp = fmaxf(z, 0.0f) + log_1to2(1.0f + e);
  sig = z >= 0.0f ? r : e * r;
}
// tanh with a short odd series near 0 (the exp form cancels there)
__device__ __forceinline__ float tanh_f(float y) {
  const float big = 1.0f - 2.0f * fast_rcp(fast_exp(2.0f * y) + 1.0f);
  const float y2 = y * y;
  const float small = y * (1.0f + y2 * (-1.0f / 3.0f + y2 * (2.0f / 15.0f + y2 * (-17.0f / 315.0f))));
  return fabsf(y) < 0.125f ? small : big;
}

// ---- input activations (queries and keys: SiLU then L2 norm; values: SiLU) --
__device__ __forceinline__ float silu_f(float x) { return x * sigmoid_f(x); }
// d SiLU / dx = sigmoid(x) (1 + x (1 - sigmoid(x)))
__device__ __forceinline__ float silu_grad_f(float x) {
  const float s = sigmoid_f(x);
  return s * (1.0f + x * (1.0f - s));
}
__device__ __forceinline__ f32x4 silu4(f32x4 x) {
  f32x4 o;
  for (int e = 0; e < 4; ++e) o[e] = silu_f(x[e]);
  return o;
}
__device__ __forceinline__ f32x4 silu_grad4(f32x4 x) {
  f32x4 o;
  for (int e = 0; e < 4; ++e) o[e] = silu_grad_f(x[e]);
  return o;
}
// the L2 normalisation is x / sqrt(|x|^2 + eps)
constexpr float kL2Eps = 1e-6f;

// sum over aligned groups of N consecutive lanes (N a power of two dividing
// 64), in every lane of the group; every lane of the wave must take part.
// Within a row of 16 lanes a DPP butterfly (lane ^ 1, lane ^ 2, then the
// half-row and row mirrors, which pair each lane with one in the other half);
// across rows lane shuffles.  Every step adds two values in either order, so
// all lanes of a group get the bitwise same sum.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N >= 1 && N <= 64 && (N & (N - 1)) == 0, "power of two up to a wave");
  if constexpr (N >= 2)
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xf, 0xf, false));
  if constexpr (N >= 4)
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x4E, 0xf, 0xf, false));
  if constexpr (N >= 8)   // row_half_mirror: lane i <-> 7 - i within each half-row
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x141, 0xf, 0xf, false));
  if constexpr (N >= 16)  // row_mirror: lane i <-> 15 - i within each row
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x140, 0xf, 0xf, false));
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

// 16 bytes of the token dtype <-> floats
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
template <typename T>
struct Chunk16;
template <>
struct Chunk16<bf16_t> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void unpack(u32x4_t v, float* f) {
    const bf16x8 b = __builtin_bit_cast(bf16x8, v);
    for (int i = 0; i < 8; ++i) f[i] = (float)b[i];
  }
  static __device__ __forceinline__ u32x4_t pack(const float* f) {
    bf16x8 b;
    for (int i = 0; i < 8; ++i) b[i] = (bf16_t)f[i];
    return __builtin_bit_cast(u32x4_t, b);
  }
};
template <>
struct Chunk16<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void unpack(u32x4_t v, float* f) {
    const f32x4 b = __builtin_bit_cast(f32x4, v);
    for (int i = 0; i < 4; ++i) f[i] = b[i];
  }
  static __device__ __forceinline__ u32x4_t pack(const float* f) {
    const f32x4 b = {f[0], f[1], f[2], f[3]};
    return __builtin_bit_cast(u32x4_t, b);
  }
};

// Sum over a row of SiLU(raw)^2, the row spread as 16-byte chunks over NC
// consecutive lanes (every lane of the wave must take part); returns
// 1 / sqrt(sum + eps), in every lane of the row.
template <typename T, int NC>
__device__ __forceinline__ float act_row_inv_norm(u32x4_t raw) {
  float f[Chunk16<T>::N];
  Chunk16<T>::unpack(raw, f);
  float ss = 0.0f;
  for (int i = 0; i < Chunk16<T>::N; ++i) {
    const float sv = silu_f(f[i]);
    ss += sv * sv;
  }
  return rsqrtf(group_sum<NC>(ss) + kL2Eps);
}
// SiLU(raw) * scale of one chunk
template <typename T>
__device__ __forceinline__ u32x4_t act_chunk(u32x4_t raw, float scale) {
  float f[Chunk16<T>::N];
  Chunk16<T>::unpack(raw, f);
  for (int i = 0; i < Chunk16<T>::N; ++i) f[i] = silu_f(f[i]) * scale;
  return Chunk16<T>::pack(f);
}

}  // namespace carve
