// carve_param.h -- the parameter-gradient partials of the CARVE backward as
// workgroup-level items: d[Ub; Uw] over a split of the chunks and dVb, dVw over
// a split of the tokens of one (batch, head); each launch of carve_bwd.hip
// runs one item per workgroup.
#pragma once
#include "carve_kernels.h"

namespace carve {

// d[Ub; Uw][r][v] = sum over the chunks of one split of sum_j dF[r][j] S_hat[v][j];
// wave w owns value tile w (S_hat read from S_chunks, lane (g, c) holding
// S_hat[16 w + c][16 jt + 4 g + e]).
// Per chunk, dF (parked as [j][r] f32) is read once with whole-row 16-byte loads
// and staged in LDS as a high and a low token-dtype part ([j][r], padded rows);
// the matrix-core operand dF[r][j] is then read with the transposing LDS load.
// SW: the scalar write gate (the fold, and dF, have the Ub rows only).
template <typename T, int D, int RF>
__host__ __device__ constexpr size_t uparam_lds() {
  return (sizeof(T) == 2 ? 2 : 1) * (size_t)D * (RF + 16 / sizeof(T)) * sizeof(T);
}

// item = (batch, head) * kUSplit + split; writes partial record `item`.  smem
// holds uparam_lds bytes; ends with a workgroup barrier.
template <typename T, int D, int RP, bool SW>
__device__ __forceinline__ void uparam_item(const BwdArgs& a, const int item, char* smem) {
  typedef Quad<T> Qd;
  typedef typename Qd::q quad;
  constexpr int NT = bwd_threads(D);
  constexpr int NJT = D / 16;
  constexpr int R2 = SW ? RP : 2 * RP;
  constexpr int NRT = R2 / 16;
  constexpr int LDR = R2 + 16 / sizeof(T);
  constexpr bool SPLIT = sizeof(T) == 2;       // f32 operands carry dF exactly
  constexpr int NV = D * R2 / 4;               // 16-byte vectors of dF
  static_assert(NV % NT == 0, "whole vectors per thread");
  T* sH = reinterpret_cast<T*>(smem);          // [D][LDR] dF rounded to T
  T* sL = sH + D * LDR;                        // [D][LDR] dF - rounded (bf16 only)
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int Tn = a.T, L = a.L, R = a.R;
  const int bh = item / kUSplit, split = item % kUSplit;
  const int nch = Tn / L;
  const ChunkRec cr = chunk_rec(sizeof(T), D, L, R2);
  const char* recb = reinterpret_cast<const char*>(a.rec) + (size_t)bh * nch * cr.total;
  f32x4 acc[NRT];
  for (int rt = 0; rt < NRT; ++rt) acc[rt] = zero4();
  const int per = (nch + kUSplit - 1) / kUSplit;
  const int c0 = split * per, c1 = c0 + per < nch ? c0 + per : nch;
  for (int ch = c0; ch < c1; ++ch) {
    const char* rc = recb + (size_t)ch * cr.total;
    const float* sv = a.S_chunks + ((size_t)bh * nch + ch) * D * D + (size_t)(16 * w + c) * D + 4 * g;
    const float* dFr = reinterpret_cast<const float*>(rc + cr.dF);
    quad sb[NJT];
    for (int jt = 0; jt < NJT; ++jt) sb[jt] = Qd::cvt(gload4(sv + 16 * jt));
    for (int u = 0; u < NV / NT; ++u) {
      const int x = tid + u * NT;
      const int j = x / (R2 / 4), r4 = (x % (R2 / 4)) * 4;
      const f32x4 v = gload4(dFr + (size_t)j * R2 + r4);
      const quad hi = Qd::cvt(v);
      Qd::st(sH + j * LDR + r4, hi);
      if (SPLIT) Qd::st(sL + j * LDR + r4, Qd::cvt(v - Qd::f32(hi)));
    }
    __syncthreads();
    for (int rt = 0; rt < NRT; ++rt)
      for (int jt = 0; jt < NJT; ++jt) {
        acc[rt] = Qd::mma16(Qd::ld_tr(sH, LDR, 16 * jt, 16 * rt, g, c), sb[jt], acc[rt]);
        if (SPLIT) acc[rt] = Qd::mma16(Qd::ld_tr(sL, LDR, 16 * jt, 16 * rt, g, c), sb[jt], acc[rt]);
      }
    __syncthreads();   // the next chunk overwrites the staged dF
  }
  float* part = a.part + (size_t)item * part_floats(R, D);
  float* pUb = part;
  float* pUw = part + (size_t)R * D;
  for (int rt = 0; rt < NRT; ++rt)
    for (int i = 0; i < 4; ++i) {
      const int rr = 16 * rt + 4 * g + i, col = 16 * w + c;
      if (rr < R) pUb[rr * D + col] = acc[rt][i];
      else if (!SW && rr >= RP && rr < RP + R) pUw[(rr - RP) * D + col] = acc[rt][i];
    }
}

// dVb[j][r] = sum_t dz_b[t][j] tau_b[t][r], dVw[v][r] = sum_t dz_w[t][v] tau_w[t][r]
// over one token split of one (batch, head); wave w owns rows 16 w .. 16 w + 15.
// The split is walked in steps of TB tokens staged through LDS (whole rows,
// 16-byte vectors); the next step's rows are loaded into registers while the
// current one is multiplied.
// SW: the scalar write gate (dVb only; tau has the b columns only).
// item = (batch, head) * kVSplit + split; writes partial record `item`.  smem
// holds vparam_lds bytes; ends with a workgroup barrier.
template <typename T>
__host__ __device__ constexpr int vparam_step_tokens() { return sizeof(T) == 2 ? 64 : 32; }

template <typename T, int D, int RP, bool SW>
__host__ __device__ constexpr size_t vparam_lds() {
  constexpr size_t PAD = 16 / sizeof(T), TB = vparam_step_tokens<T>();
  return (2 * TB * (D + PAD) + TB * ((SW ? RP : 2 * RP) + PAD)) * sizeof(T);
}

template <typename T, int D, int RP, bool SW>
__device__ __forceinline__ void vparam_item(const BwdArgs& a, const int item, char* smem) {
  typedef Quad<T> Qd;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr int NT = bwd_threads(D);
  constexpr int R2 = SW ? RP : 2 * RP;
  constexpr int NRB = RP / 16;
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDD = D + PAD, LDR = R2 + PAD;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int TB = vparam_step_tokens<T>();
  constexpr int NC = D / VEC, NCR = R2 / VEC;            // 16-byte vectors per token / tau row
  constexpr int NVT = (TB * NC + NT - 1) / NT, NTT = (TB * NCR + NT - 1) / NT;
  T* sB = reinterpret_cast<T*>(smem);          // [TB][LDD] dz_b of a step
  T* sW = sB + TB * LDD;                       // [TB][LDD] dz_w of a step
  T* sTau = sW + TB * LDD;                     // [TB][LDR] tau of the step

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int H = a.H, Tn = a.T, L = a.L, R = a.R;
  const int bh = item / kVSplit, split = item % kVSplit;
  const int b = bh / H, h = bh % H;
  const int nch = Tn / L;
  const size_t bh0 = ((size_t)b * Tn * H + h) * D;
  const int rs = H * D;
  const T* __restrict__ dbx = reinterpret_cast<const T*>(a.dbx) + bh0;
  const T* __restrict__ dwx = reinterpret_cast<const T*>(a.dwx) + bh0;
  const ChunkRec cr = chunk_rec(sizeof(T), D, L, R2);
  const char* recb = reinterpret_cast<const char*>(a.rec) + (size_t)bh * nch * cr.total;

  f32x4 accB[NRB], accW[NRB];
  for (int rt = 0; rt < NRB; ++rt) { accB[rt] = zero4(); accW[rt] = zero4(); }
  const int nblk = Tn / 16;
  const int per = (nblk + kVSplit - 1) / kVSplit;
  const int blk0 = split * per, blk1 = blk0 + per < nblk ? blk0 + per : nblk;
  const int t_begin = 16 * blk0, t_end = 16 * blk1;
  u32x4 pb[NVT], pw[NVT], pt[NTT];
  // rows of tokens t0 .. t0 + nt - 1 into registers (vector x of a step: token
  // x / NC, elements (x % NC) * VEC ..; tau rows from the chunk records)
  auto load = [&](const int t0) {
    const int nt = t_end - t0 < TB ? t_end - t0 : TB;
    for (int u = 0; u < NVT; ++u) {
      const int x = tid + u * NT;
      if (x < nt * NC) {
        const int o = (t0 + x / NC) * rs + (x % NC) * VEC;
        pb[u] = *reinterpret_cast<const u32x4*>(dbx + o);
        if constexpr (!SW) pw[u] = *reinterpret_cast<const u32x4*>(dwx + o);
      }
    }
    for (int u = 0; u < NTT; ++u) {
      const int x = tid + u * NT;
      if (x < nt * NCR) {
        const int tt = t0 + x / NCR;
        const T* tau = reinterpret_cast<const T*>(recb + (size_t)(tt / L) * cr.total + cr.Tau);
        pt[u] = *reinterpret_cast<const u32x4*>(tau + (tt % L) * R2 + (x % NCR) * VEC);
      }
    }
  };
  auto stage = [&](const int t0) {
    const int nt = t_end - t0 < TB ? t_end - t0 : TB;
    for (int u = 0; u < NVT; ++u) {
      const int x = tid + u * NT;
      if (x < nt * NC) {
        const int o = (x / NC) * LDD + (x % NC) * VEC;
        *reinterpret_cast<u32x4*>(sB + o) = pb[u];
        if constexpr (!SW) *reinterpret_cast<u32x4*>(sW + o) = pw[u];
      }
    }
    for (int u = 0; u < NTT; ++u) {
      const int x = tid + u * NT;
      if (x < nt * NCR) *reinterpret_cast<u32x4*>(sTau + (x / NCR) * LDR + (x % NCR) * VEC) = pt[u];
    }
  };
  if (t_begin < t_end) load(t_begin);
  for (int t0 = t_begin; t0 < t_end; t0 += TB) {
    stage(t0);
    if (t0 + TB < t_end) load(t0 + TB);
    __syncthreads();
    const int nb = (t_end - t0 < TB ? t_end - t0 : TB) / 16;
    for (int bb = 0; bb < nb; ++bb) {
      // lane (g, c): dz_b[t = 16 bb + 4 g + e][j = 16 w + c]
      const typename Qd::q ab = Qd::ld_tr(sB + bb * 16 * LDD, LDD, 0, 16 * w, g, c);
      for (int rt = 0; rt < NRB; ++rt)
        accB[rt] = Qd::mma16(ab, Qd::ld_tr(sTau + bb * 16 * LDR, LDR, 0, 16 * rt, g, c), accB[rt]);
      if constexpr (!SW) {
        const typename Qd::q aw = Qd::ld_tr(sW + bb * 16 * LDD, LDD, 0, 16 * w, g, c);
        for (int rt = 0; rt < NRB; ++rt)
          accW[rt] = Qd::mma16(aw, Qd::ld_tr(sTau + bb * 16 * LDR, LDR, 0, RP + 16 * rt, g, c), accW[rt]);
      }
    }
    __syncthreads();
  }
  float* part = a.partV + (size_t)item * part_floats(R, D);
  for (int rt = 0; rt < NRB; ++rt)
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * w + 4 * g + i, col = 16 * rt + c;
      if (col < R) {
        part[row * R + col] = accB[rt][i];
        if constexpr (!SW) part[(size_t)R * D + row * R + col] = accW[rt][i];
      }
    }
}

}  // namespace carve
