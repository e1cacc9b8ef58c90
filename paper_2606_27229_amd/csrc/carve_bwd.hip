// carve_bwd.hip -- chunked CARVE backward on gfx950.
//
// One workgroup per (batch, head) walks the gate chunks in reverse (App. Alg.
// megakernel_bwd).  The state gradient dS (Dv x Dk, f32) stays in registers
// for the whole call in the same layout as the forward state: wave w owns key
// columns [16w, 16w+16) for every value row.
//
// Per gate chunk c:
//   S_hat = S_chunks[c] (written by the forward), F = [Ub; Uw] S_hat (fold).
//   If the chunk holds several 16-token WY tiles, the tile start states are
//   recomputed by running the forward tiles once and parked in the workspace.
//   Then per 16-token tile, last to first, with S the tile start state and dS'
//   the gradient of the tile end state:
//     recompute tau, gates, Lam (inclusive prefix sums of l = g - softplus(z_b)),
//       E = e^{Lam}, E' = e^{Lam_{t-1}}, en = e^{-Lam}, gam = e^{Lam_15},
//       A = beta D with D_ts = (k E')_t . (k en)_s (s < t), P_ts = (q E)_t . (k en)_s
//       (s <= t), T = (I + A)^{-1}, R = beta (w v - Ktil S^T), u = T R
//     adjoint (the tile's forward is S' = S diag(gam) + u^T Khat, O = Qtil S^T + P u):
//       du  = Khat dS'^T + P^T dO,   dR = T^T du,   dE = beta dR
//       dw  = dE * v,  dv = dE * w,  dz_w = dw w (1 - w)
//       dKtil = -dE S, dQtil = dO S, dKhat = u dS'
//       dP  = dO u^T (s <= t), dA = -dR u^T (s < t), dD = beta dA
//       dbeta = rowsum(dR * (w v - Ktil S^T)) + rowsum(dA * D)
//       k/q gradients through the factored pair products, and dLam from the
//       identity d/dLam of e^{Lam_a - Lam_b} = +/- the term itself
//       dl = reverse prefix sums of dLam;  dg = dl;  dz_b = -dl b
//       dtau = dz V;  dY = dtau (1 - tau^2);  dq += dY F;  dF += dY^T q
//       dVb += dz_b^T tau_b, dVw += dz_w^T tau_w
//       dS <- dS' diag(gam) + dO^T Qtil - dE^T Ktil
//   At the chunk start the folded read-out closes the chain ("glue"):
//       dS += [Ub; Uw]^T dF,   d[Ub; Uw] += dF S_hat^T.
// Parameter gradients are kept per (batch, head) and reduced afterwards in a
// fixed order (carve_param_reduce), so reruns are bitwise identical.
#include "carve_kernels.h"

namespace carve {

constexpr int BLW = 16;  // WY tile of the backward

struct BwdLds {
  size_t S, dS, F, Q, K, Ki, QT, KT, KiT, Tau, A, Dm, Tb, TbT, PT, RT, U, UTz, KhTz, dO, dOT, duT,
      dR, dE, dET, dD, dDT, dP, dPT, dY, dYT, Gam, Beta, Db, Db2, total;
};

template <typename T, int D>
__host__ __device__ constexpr BwdLds bwd_lds(int RP) {
  BwdLds l{};
  size_t off = 0;
  const size_t e = sizeof(T);
  const size_t R2 = 2 * (size_t)RP;
  constexpr size_t LD = (size_t)BLW * D;   // [16][D] or [D][16]
  constexpr size_t LL = (size_t)BLW * BLW; // [16][16]
  l.S = off;    off += lds_round((size_t)D * D * e);
  l.dS = off;   off += lds_round((size_t)D * D * e);
  l.F = off;    off += lds_round(R2 * D * e);
  // transient region; dF (R2 x D) for the parameter product at a chunk start
  // reuses it once the tiles of the chunk are done
  l.Q = off;    off += lds_round(LD * e);
  l.K = off;    off += lds_round(LD * e);
  l.Ki = off;   off += lds_round(LD * e);
  l.QT = off;   off += lds_round(LD * e);
  l.KT = off;   off += lds_round(LD * e);
  l.KiT = off;  off += lds_round(LD * e);
  l.Tau = off;  off += lds_round((size_t)BLW * R2 * e);
  l.A = off;    off += lds_round(LL * 4);
  l.Dm = off;   off += lds_round(LL * 4);
  l.Tb = off;   off += lds_round(LL * e);
  l.TbT = off;  off += lds_round(LL * e);
  l.PT = off;   off += lds_round(LL * e);
  l.RT = off;   off += lds_round(LD * e);
  l.U = off;    off += lds_round(LD * e);
  l.UTz = off;  off += lds_round(LD * e);   // u^T (forward tiles) / dz_b (backward tiles)
  l.KhTz = off; off += lds_round(LD * e);   // Khat^T (forward tiles) / dz_w (backward tiles)
  l.dO = off;   off += lds_round(LD * e);
  l.dOT = off;  off += lds_round(LD * e);
  l.duT = off;  off += lds_round(LD * e);
  l.dR = off;   off += lds_round(LD * e);
  l.dE = off;   off += lds_round(LD * e);
  l.dET = off;  off += lds_round(LD * e);
  l.dD = off;   off += lds_round(LL * e);
  l.dDT = off;  off += lds_round(LL * e);
  l.dP = off;   off += lds_round(LL * e);
  l.dPT = off;  off += lds_round(LL * e);
  l.dY = off;   off += lds_round((size_t)BLW * R2 * e);
  l.dYT = off;  off += lds_round((size_t)BLW * R2 * e);
  l.Gam = off;  off += lds_round((size_t)D * 4);
  l.Beta = off; off += lds_round((size_t)BLW * 4);
  l.Db = off;   off += lds_round((size_t)(D / 16) * BLW * 4);
  l.Db2 = off;  off += lds_round((size_t)BLW * 4);
  l.total = off;
  return l;
}

// acc += A[0:16 rows][0:16] . B[..][0:16]^T for a K = 16 token contraction;
// a_row / b_row point at this lane's row (K-contiguous).  bf16 uses one
// 16x16x32 instruction with the upper half of K zero.
template <typename T>
__device__ __forceinline__ f32x4 mma_k16(f32x4 acc, const T* a_row, const T* b_row, int g) {
  typedef Mma<T> M;
  if constexpr (sizeof(T) == 2) {
    const typename M::frag a = g < 2 ? M::load(a_row + 8 * g) : M::zero();
    const typename M::frag b = g < 2 ? M::load(b_row + 8 * g) : M::zero();
    acc = M::mma(a, b, acc);
  } else {
    for (int ks = 0; ks < 4; ++ks) acc = M::mma(a_row[4 * ks + g], b_row[4 * ks + g], acc);
  }
  return acc;
}

// acc += A . Reg where the contraction runs over the rows of a D x 16 column
// block held in registers (Reg[it][r] = X[16 it + 4g + r][col c]); a_row is
// this lane's row of A, K-contiguous over those D rows.  The K slots are
// permuted identically on both operands.
template <typename T, int NIT>
__device__ __forceinline__ f32x4 mma_regB(f32x4 acc, const T* a_row, const f32x4* Reg, int g) {
  typedef Mma<T> M;
  if constexpr (sizeof(T) == 2) {
    for (int ks = 0; ks < NIT / 2; ++ks) {
      typename M::frag a, b;
      const T* p = a_row + 32 * ks + 4 * g;
      for (int e = 0; e < 4; ++e) {
        a[e] = p[e];
        a[4 + e] = p[16 + e];
        b[e] = (T)Reg[2 * ks][e];
        b[4 + e] = (T)Reg[2 * ks + 1][e];
      }
      acc = M::mma(a, b, acc);
    }
  } else {
    for (int it = 0; it < NIT; ++it)
      for (int r = 0; r < 4; ++r) acc = M::mma(a_row[16 * it + 4 * g + r], Reg[it][r], acc);
  }
  return acc;
}

template <typename T, int D>
__global__ void __launch_bounds__(D * 4) carve_bwd_kernel(BwdArgs a) {
  typedef Mma<T> M;
  constexpr int NW = D / 16;
  constexpr int NT = NW * 64;
  constexpr int NIT = D / 16;
  constexpr int KS = M::KS, KPL = M::KPL;
  const int RP = a.RP, R2 = 2 * a.RP, R = a.R;
  const int H = a.H, Tn = a.T, L = a.L;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int nch = Tn / L, msub = L / BLW;
  const int jj = 16 * w + c;  // this lane's key column / value column

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const BwdLds lay = bwd_lds<T, D>(RP);
  T* sS = reinterpret_cast<T*>(smem + lay.S);
  T* sdS = reinterpret_cast<T*>(smem + lay.dS);
  T* sF = reinterpret_cast<T*>(smem + lay.F);
  T* sQ = reinterpret_cast<T*>(smem + lay.Q);
  T* sK = reinterpret_cast<T*>(smem + lay.K);
  T* sKi = reinterpret_cast<T*>(smem + lay.Ki);
  T* sQT = reinterpret_cast<T*>(smem + lay.QT);
  T* sKT = reinterpret_cast<T*>(smem + lay.KT);
  T* sKiT = reinterpret_cast<T*>(smem + lay.KiT);
  T* sTau = reinterpret_cast<T*>(smem + lay.Tau);
  float* sA = reinterpret_cast<float*>(smem + lay.A);
  float* sDm = reinterpret_cast<float*>(smem + lay.Dm);
  T* sTb = reinterpret_cast<T*>(smem + lay.Tb);
  T* sTbT = reinterpret_cast<T*>(smem + lay.TbT);
  T* sPT = reinterpret_cast<T*>(smem + lay.PT);
  T* sRT = reinterpret_cast<T*>(smem + lay.RT);
  T* sU = reinterpret_cast<T*>(smem + lay.U);
  T* sUT = reinterpret_cast<T*>(smem + lay.UTz);
  T* sdzb = sUT;
  T* sKhT = reinterpret_cast<T*>(smem + lay.KhTz);
  T* sdzw = sKhT;
  T* sdO = reinterpret_cast<T*>(smem + lay.dO);
  T* sdOT = reinterpret_cast<T*>(smem + lay.dOT);
  T* sduT = reinterpret_cast<T*>(smem + lay.duT);
  T* sdR = reinterpret_cast<T*>(smem + lay.dR);
  T* sdE = reinterpret_cast<T*>(smem + lay.dE);
  T* sdET = reinterpret_cast<T*>(smem + lay.dET);
  T* sdD = reinterpret_cast<T*>(smem + lay.dD);
  T* sdDT = reinterpret_cast<T*>(smem + lay.dDT);
  T* sdP = reinterpret_cast<T*>(smem + lay.dP);
  T* sdPT = reinterpret_cast<T*>(smem + lay.dPT);
  T* sdY = reinterpret_cast<T*>(smem + lay.dY);
  T* sdYT = reinterpret_cast<T*>(smem + lay.dYT);
  float* sGam = reinterpret_cast<float*>(smem + lay.Gam);
  float* sBeta = reinterpret_cast<float*>(smem + lay.Beta);
  float* sDb = reinterpret_cast<float*>(smem + lay.Db);
  float* sDb2 = reinterpret_cast<float*>(smem + lay.Db2);
  T* sdF = sQ;  // [R2][D] at a chunk start; the transient region is free then

  const T* __restrict__ q = reinterpret_cast<const T*>(a.q);
  const T* __restrict__ k = reinterpret_cast<const T*>(a.k);
  const T* __restrict__ v = reinterpret_cast<const T*>(a.v);
  const T* __restrict__ bx = reinterpret_cast<const T*>(a.bx);
  const T* __restrict__ wx = reinterpret_cast<const T*>(a.wx);
  const T* __restrict__ beta = reinterpret_cast<const T*>(a.beta);
  const T* __restrict__ dO = reinterpret_cast<const T*>(a.dO);
  T* __restrict__ dq = reinterpret_cast<T*>(a.dq);
  T* __restrict__ dk = reinterpret_cast<T*>(a.dk);
  T* __restrict__ dv = reinterpret_cast<T*>(a.dv);
  T* __restrict__ dbeta = reinterpret_cast<T*>(a.dbeta);
  T* __restrict__ dbx = reinterpret_cast<T*>(a.dbx);
  T* __restrict__ dwx = reinterpret_cast<T*>(a.dwx);

  const size_t soff = (size_t)bh * D * D;
  float* part = a.part + (size_t)bh * part_floats(R, D);
  float* pUb = part;
  float* pUw = part + (size_t)R * D;
  float* pVb = part + (size_t)2 * R * D;
  float* pVw = part + (size_t)3 * R * D;
  // clear the dUcat entries this lane accumulates at every chunk start
  for (int rt = 0; rt < R2 / 16; ++rt)
    for (int r = 0; r < 4; ++r) {
      const int rr = 16 * rt + 4 * g + r;
      if (rr < R) pUb[(size_t)rr * D + jj] = 0.0f;
      else if (rr >= RP && rr < RP + R) pUw[(size_t)(rr - RP) * D + jj] = 0.0f;
    }

  f32x4 S[NIT], dS[NIT], dF[8], dVb[4], dVw[4];  // R2/16 <= 8, RP/16 <= 4
  for (int it = 0; it < NIT; ++it)
    for (int r = 0; r < 4; ++r)
      dS[it][r] = a.dS_T ? a.dS_T[soff + (size_t)(16 * it + 4 * g + r) * D + jj] : 0.0f;
  for (int x = 0; x < 4; ++x) {
    dVb[x] = zero4();
    dVw[x] = zero4();
  }

  for (int ch = nch - 1; ch >= 0; --ch) {
    const float* Shat = a.S_chunks + ((size_t)bh * nch + ch) * D * D;
    for (int it = 0; it < NIT; ++it)
      for (int r = 0; r < 4; ++r) S[it][r] = Shat[(size_t)(16 * it + 4 * g + r) * D + jj];
    for (int x = 0; x < 8; ++x) dF[x] = zero4();
    // fold F = [Ub; Uw] S_hat -> sF [R2][D]
    __syncthreads();
    for (int rt = 0; rt < R2 / 16; ++rt) {
      const int rr = 16 * rt + c;
      const float* urow = nullptr;
      if (rr < R) urow = a.Ub + (size_t)rr * D;
      else if (rr >= RP && rr < RP + R) urow = a.Uw + (size_t)(rr - RP) * D;
      f32x4 acc = zero4();
      if constexpr (KPL == 8) {
        for (int ks = 0; ks < D / 32; ++ks) {
          typename M::frag af, bfg;
          const int i0 = 32 * ks + 4 * g;
          for (int e = 0; e < 4; ++e) {
            af[e] = (T)S[2 * ks][e];
            af[4 + e] = (T)S[2 * ks + 1][e];
            bfg[e] = (T)(urow ? urow[i0 + e] : 0.0f);
            bfg[4 + e] = (T)(urow ? urow[i0 + 16 + e] : 0.0f);
          }
          acc = M::mma(af, bfg, acc);
        }
      } else {
        for (int it = 0; it < NIT; ++it)
          for (int r4 = 0; r4 < 4; ++r4) {
            const float bv = urow ? urow[16 * it + 4 * g + r4] : 0.0f;
            acc = M::mma((T)S[it][r4], (T)bv, acc);
          }
      }
      store_tile_t(sF, D, 16 * w, 16 * rt, acc, lane);
    }

    // pass 0: forward tiles 0..msub-2 recompute the tile start states;
    // pass 1: backward tiles msub-1..0
    for (int pass = (msub > 1 ? 0 : 1); pass < 2; ++pass) {
      const bool bwd = pass == 1;
      const int mcount = bwd ? msub : msub - 1;
      for (int mi = 0; mi < mcount; ++mi) {
        const int m = bwd ? (msub - 1 - mi) : mi;
        const int t0 = ch * L + m * BLW;
        const size_t tokbase = ((size_t)b * Tn + t0) * H + h;
        if (bwd && msub > 1) {
          const float* src = (m == 0) ? Shat : a.substates + ((size_t)bh * msub + m) * D * D;
          for (int it = 0; it < NIT; ++it)
            for (int r = 0; r < 4; ++r) S[it][r] = src[(size_t)(16 * it + 4 * g + r) * D + jj];
        }
        __syncthreads();  // previous users of the transient buffers are done
        // ---- B0: loads --------------------------------------------------------
        {
          constexpr int VEC = 16 / sizeof(T);
          constexpr int NV = BLW * D / VEC;
          for (int x = tid; x < NV; x += NT) {
            const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;
            const size_t gofs = (tokbase + (size_t)t * H) * D + j;
            *reinterpret_cast<f32x4*>(sQ + t * D + j) = *reinterpret_cast<const f32x4*>(q + gofs);
            *reinterpret_cast<f32x4*>(sK + t * D + j) = *reinterpret_cast<const f32x4*>(k + gofs);
            if (bwd) {
              const f32x4 raw = *reinterpret_cast<const f32x4*>(dO + gofs);
              *reinterpret_cast<f32x4*>(sdO + t * D + j) = raw;
              const T* rv = reinterpret_cast<const T*>(&raw);
              for (int e = 0; e < VEC; ++e) sdOT[(j + e) * BLW + t] = rv[e];
            }
          }
          if (tid < BLW) sBeta[tid] = to_f(beta[tokbase + (size_t)tid * H]);
          for (int it = 0; it < NIT; ++it) {
            store_tile(sS, D, 16 * it, 16 * w, S[it], lane);
            if (bwd) store_tile(sdS, D, 16 * it, 16 * w, dS[it], lane);
          }
        }
        __syncthreads();
        // ---- R1: tau = tanh(Q F^T) --------------------------------------------
        for (int rt = w; rt < R2 / 16; rt += NW) {
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sQ + c * D + kofs), M::load(sF + (16 * rt + c) * D + kofs), acc);
          }
          for (int r = 0; r < 4; ++r) acc[r] = tanh_f(acc[r]);
          store_tile(sTau, R2, 0, 16 * rt, acc, lane);
        }
        __syncthreads();
        // ---- R2: gates and retention factors ------------------------------------
        float qv[4], kv[4], E[4], Ep[4], en[4], bgt[4], wgt[4], vv[4], wv[4];
        float gam;
        {
          f32x4 accB = zero4(), accW = zero4();
          for (int ks = 0; ks < RP / KS; ++ks) {
            const int r0 = ks * KS + g * KPL;
            float vb[KPL], vw[KPL];
            for (int e = 0; e < KPL; ++e) {
              const int rr = r0 + e;
              vb[e] = rr < R ? a.Vb[(size_t)jj * R + rr] : 0.0f;
              vw[e] = rr < R ? a.Vw[(size_t)jj * R + rr] : 0.0f;
            }
            accB = M::mma(M::load(sTau + c * R2 + r0), M::from_f32(vb), accB);
            accW = M::mma(M::load(sTau + c * R2 + RP + r0), M::from_f32(vw), accW);
          }
          float p[4];
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            const size_t e = (tokbase + (size_t)t * H) * D + jj;
            const float zb = to_f(bx[e]) + accB[r];
            p[r] = a.g[e] - softplus_f(zb);
            bgt[r] = sigmoid_f(zb);
            wgt[r] = sigmoid_f(to_f(wx[e]) + accW[r]);
            vv[r] = to_f(v[e]);
            wv[r] = wgt[r] * vv[r];
            qv[r] = to_f(sQ[t * D + jj]);
            kv[r] = to_f(sK[t * D + jj]);
          }
          p[1] += p[0];
          p[2] += p[1];
          p[3] += p[2];
          float incl = p[3];
          float y = __shfl_up(incl, 16);
          if (g >= 1) incl += y;
          y = __shfl_up(incl, 32);
          if (g >= 2) incl += y;
          const float excl = incl - p[3];
          const float lam_end = __shfl(incl, 48 + c);
          for (int r = 0; r < 4; ++r) {
            const float lam = excl + p[r];
            E[r] = fast_exp(lam);
            en[r] = fast_exp(-lam);
          }
          const float eprev = __shfl_up(E[3], 16);
          Ep[0] = g == 0 ? 1.0f : eprev;
          Ep[1] = E[0];
          Ep[2] = E[1];
          Ep[3] = E[2];
          gam = fast_exp(lam_end);
          f32x4 vK, vQ, vKi, vKh;
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            vK[r] = kv[r] * Ep[r];
            vQ[r] = qv[r] * E[r];
            vKi[r] = kv[r] * en[r];
            vKh[r] = vKi[r] * gam;
            sK[t * D + jj] = (T)vK[r];
            sQ[t * D + jj] = (T)vQ[r];
            sKi[t * D + jj] = (T)vKi[r];
          }
          store_tile_t(sKT, BLW, 0, 16 * w, vK, lane);
          store_tile_t(sQT, BLW, 0, 16 * w, vQ, lane);
          store_tile_t(sKiT, BLW, 0, 16 * w, vKi, lane);
          if (!bwd) store_tile_t(sKhT, BLW, 0, 16 * w, vKh, lane);
          if (g == 0) sGam[jj] = gam;
        }
        __syncthreads();
        // ---- R3: A, D, P and Ktil S^T --------------------------------------------
        if (w == 0) {
          f32x4 accA = zero4(), accP = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            const typename M::frag kb = M::load(sKi + c * D + kofs);
            accA = M::mma(M::load(sK + c * D + kofs), kb, accA);
            accP = M::mma(M::load(sQ + c * D + kofs), kb, accP);
          }
          f32x4 pv;
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            const float dval = (c < t) ? accA[r] : 0.0f;
            sDm[t * BLW + c] = dval;
            sA[t * BLW + c] = sBeta[t] * dval;
            pv[r] = (c <= t) ? accP[r] : 0.0f;
          }
          store_tile_t(sPT, BLW, 0, 0, pv, lane);
        }
        float Eerr[4];
        {
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sK + c * D + kofs), M::load(sS + (16 * w + c) * D + kofs), acc);
          }
          f32x4 rv;
          for (int r = 0; r < 4; ++r) {
            Eerr[r] = wv[r] - acc[r];
            rv[r] = sBeta[4 * g + r] * Eerr[r];
          }
          store_tile_t(sRT, BLW, 0, 16 * w, rv, lane);
        }
        __syncthreads();
        // ---- R4: T = (I + A)^{-1}; du = Khat dS'^T + P^T dO ----------------------
        if (w == 0 && g == 0) {
          float x[16];
#pragma unroll
          for (int t = 0; t < 16; ++t) {
            float acc = (t == c) ? 1.0f : 0.0f;
#pragma unroll
            for (int s = 0; s < t; ++s) acc -= sA[t * BLW + s] * x[s];
            x[t] = acc;
          }
#pragma unroll
          for (int t = 0; t < 16; ++t) {
            sTb[t * BLW + c] = (T)x[t];
            sTbT[c * BLW + t] = (T)x[t];
          }
        }
        if (bwd) {
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load_scaled(sKi + c * D + kofs, sGam + kofs), M::load(sdS + (16 * w + c) * D + kofs), acc);
          }
          acc = mma_k16<T>(acc, sPT + c * BLW, sdOT + (16 * w + c) * BLW, g);
          store_tile_t(sduT, BLW, 0, 16 * w, acc, lane);
        }
        __syncthreads();
        // ---- R5: u = T R; dR = T^T du ---------------------------------------------
        float dzw[4];
        {
          const f32x4 u = mma_k16<T>(zero4(), sTb + c * BLW, sRT + (16 * w + c) * BLW, g);
          if (bwd) {
            store_tile(sU, D, 0, 16 * w, u, lane);
            const f32x4 dR = mma_k16<T>(zero4(), sTbT + c * BLW, sduT + (16 * w + c) * BLW, g);
            f32x4 dE, dzv;
            for (int r = 0; r < 4; ++r) {
              const int t = 4 * g + r;
              dE[r] = sBeta[t] * dR[r];
              float db = dR[r] * Eerr[r];
              db += __shfl_xor(db, 1);
              db += __shfl_xor(db, 2);
              db += __shfl_xor(db, 4);
              db += __shfl_xor(db, 8);
              if (c == 0) sDb[w * BLW + t] = db;
              const float dwv = dE[r] * vv[r];
              const size_t e = (tokbase + (size_t)t * H) * D + jj;
              dv[e] = (T)(dE[r] * wgt[r]);
              dzw[r] = dwv * wgt[r] * (1.0f - wgt[r]);
              dwx[e] = (T)dzw[r];
              dzv[r] = dzw[r];
            }
            store_tile(sdR, D, 0, 16 * w, dR, lane);
            store_tile(sdE, D, 0, 16 * w, dE, lane);
            store_tile_t(sdET, BLW, 0, 16 * w, dE, lane);
            store_tile(sdzw, D, 0, 16 * w, dzv, lane);
          } else {
            store_tile_t(sUT, BLW, 0, 16 * w, u, lane);
          }
        }
        __syncthreads();
        if (!bwd) {
          // forward tile: S <- S diag(gam) + u^T Khat, park it for the backward tiles
          float* dst = a.substates + ((size_t)bh * msub + m + 1) * D * D;
          for (int it = 0; it < NIT; ++it) {
            f32x4 acc;
            for (int r = 0; r < 4; ++r) acc[r] = S[it][r] * gam;
            acc = mma_k16<T>(acc, sUT + (16 * it + c) * BLW, sKhT + (16 * w + c) * BLW, g);
            S[it] = acc;
            for (int r = 0; r < 4; ++r) dst[(size_t)(16 * it + 4 * g + r) * D + jj] = acc[r];
          }
          continue;
        }
        // ---- G3: dKtil = -dE S, dQtil = dO S, dKhat = u dS'; dP, dA -------------
        f32x4 dKt = mma_regB<T, NIT>(zero4(), sdE + c * D, S, g);
        for (int r = 0; r < 4; ++r) dKt[r] = -dKt[r];
        f32x4 dQt = mma_regB<T, NIT>(zero4(), sdO + c * D, S, g);
        f32x4 dKh = mma_regB<T, NIT>(zero4(), sU + c * D, dS, g);
        float cs = 0.0f;  // colsum(S * dS') for column jj
        for (int it = 0; it < NIT; ++it)
          for (int r = 0; r < 4; ++r) cs += S[it][r] * dS[it][r];
        cs += __shfl_xor(cs, 16);
        cs += __shfl_xor(cs, 32);
        if (w == 0) {
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sdO + c * D + kofs), M::load(sU + c * D + kofs), acc);
          }
          for (int r = 0; r < 4; ++r) acc[r] = (c <= 4 * g + r) ? acc[r] : 0.0f;
          store_tile(sdP, BLW, 0, 0, acc, lane);
          store_tile_t(sdPT, BLW, 0, 0, acc, lane);
        }
        if (w == (NW > 1 ? 1 : 0)) {
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sdR + c * D + kofs), M::load(sU + c * D + kofs), acc);
          }
          f32x4 ddv;
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            const float dA = (c < t) ? -acc[r] : 0.0f;
            ddv[r] = sBeta[t] * dA;
            float db = dA * sDm[t * BLW + c];
            db += __shfl_xor(db, 1);
            db += __shfl_xor(db, 2);
            db += __shfl_xor(db, 4);
            db += __shfl_xor(db, 8);
            if (c == 0) sDb2[t] = db;
          }
          store_tile(sdD, BLW, 0, 0, ddv, lane);
          store_tile_t(sdDT, BLW, 0, 0, ddv, lane);
        }
        __syncthreads();
        // ---- G5: factored-pair gradients, dLam, gate-logit gradients -------------
        float dqv[4], dkv[4];
        {
          const f32x4 dAq = mma_k16<T>(zero4(), sdD + c * BLW, sKiT + (16 * w + c) * BLW, g);
          const f32x4 dPq = mma_k16<T>(zero4(), sdP + c * BLW, sKiT + (16 * w + c) * BLW, g);
          f32x4 dcol = mma_k16<T>(zero4(), sdDT + c * BLW, sKT + (16 * w + c) * BLW, g);
          dcol = mma_k16<T>(dcol, sdPT + c * BLW, sQT + (16 * w + c) * BLW, g);
          float aL[4], pL[4], xs = 0.0f;
          for (int r = 0; r < 4; ++r) {
            const float gq = dQt[r] * E[r] + E[r] * dPq[r];          // dq from Qtil and P
            const float gkh = dKh[r] * gam * en[r];                  // dk from Khat
            const float gkc = en[r] * dcol[r];                       // dk from the column side
            const float gkr = dKt[r] * Ep[r] + Ep[r] * dAq[r];       // dk from Ktil and the row side of A
            dqv[r] = gq;
            dkv[r] = gkr + gkh + gkc;
            aL[r] = qv[r] * gq - kv[r] * gkc - kv[r] * gkh;
            pL[r] = kv[r] * gkr;
            xs += kv[r] * gkh;
          }
          xs += __shfl_xor(xs, 16);
          xs += __shfl_xor(xs, 32);
          if (g == 3) aL[3] += xs + cs * gam;
          const float pnext = __shfl_down(pL[0], 16);
          float dLam[4];
          dLam[0] = aL[0] + pL[1];
          dLam[1] = aL[1] + pL[2];
          dLam[2] = aL[2] + pL[3];
          dLam[3] = aL[3] + (g < 3 ? pnext : 0.0f);
          // reverse prefix sums over the 16 rows
          float sfx[4];
          sfx[3] = dLam[3];
          sfx[2] = sfx[3] + dLam[2];
          sfx[1] = sfx[2] + dLam[1];
          sfx[0] = sfx[1] + dLam[0];
          float tot = sfx[0];
          float z = __shfl_down(tot, 16);
          if (g <= 2) tot += z;
          z = __shfl_down(tot, 32);
          if (g <= 1) tot += z;
          const float after = tot - sfx[0];  // sum over the rows of later lane groups
          f32x4 dzb;
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            const float dl = sfx[r] + after;
            const size_t e = (tokbase + (size_t)t * H) * D + jj;
            a.dg[e] = dl;
            dzb[r] = -dl * bgt[r];
            dbx[e] = (T)dzb[r];
          }
          store_tile(sdzb, D, 0, 16 * w, dzb, lane);
          // dVb += dz_b^T tau_b, dVw += dz_w^T tau_w (A from registers, K = 16 tokens)
          for (int rt = 0; rt < RP / 16; ++rt) {
            if constexpr (sizeof(T) == 2) {
              typename M::frag ab, aw, bb, bw;
              for (int e = 0; e < 4; ++e) {
                ab[e] = (T)dzb[e];
                aw[e] = (T)dzw[e];
                bb[e] = sTau[(4 * g + e) * R2 + 16 * rt + c];
                bw[e] = sTau[(4 * g + e) * R2 + RP + 16 * rt + c];
                ab[4 + e] = (T)0.0f;
                aw[4 + e] = (T)0.0f;
                bb[4 + e] = (T)0.0f;
                bw[4 + e] = (T)0.0f;
              }
              dVb[rt] = M::mma(ab, bb, dVb[rt]);
              dVw[rt] = M::mma(aw, bw, dVw[rt]);
            } else {
              for (int r = 0; r < 4; ++r) {
                dVb[rt] = M::mma(dzb[r], sTau[(4 * g + r) * R2 + 16 * rt + c], dVb[rt]);
                dVw[rt] = M::mma(dzw[r], sTau[(4 * g + r) * R2 + RP + 16 * rt + c], dVw[rt]);
              }
            }
          }
        }
        __syncthreads();
        // ---- G8: dtau = dz V, dY = dtau (1 - tau^2) ------------------------------
        for (int x = w; x < 2 * (RP / 16); x += NW) {
          const int half = x / (RP / 16), rt = x % (RP / 16);
          const T* arow = (half ? sdzw : sdzb) + c * D;
          const float* Vm = half ? a.Vw : a.Vb;
          const int col = 16 * rt + c;  // column of V this lane supplies
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int j0 = ks * KS + g * KPL;
            float vb[KPL];
            for (int e = 0; e < KPL; ++e) vb[e] = col < R ? Vm[(size_t)(j0 + e) * R + col] : 0.0f;
            acc = M::mma(M::load(arow + j0), M::from_f32(vb), acc);
          }
          f32x4 dy;
          for (int r = 0; r < 4; ++r) {
            const float tv = to_f(sTau[(4 * g + r) * R2 + half * RP + 16 * rt + c]);
            dy[r] = acc[r] * (1.0f - tv * tv);
          }
          store_tile(sdY, R2, 0, half * RP + 16 * rt, dy, lane);
          store_tile_t(sdYT, BLW, 0, half * RP + 16 * rt, dy, lane);
        }
        __syncthreads();
        // ---- G9: dq += dY F, outputs, dF += dY^T q, dS <- ... ---------------------
        {
          f32x4 acc = zero4();
          for (int ks = 0; ks < R2 / KS; ++ks) {
            const int r0 = ks * KS + g * KPL;
            typename M::frag bfg;
            if constexpr (KPL == 8) {
              for (int e = 0; e < 8; ++e) bfg[e] = sF[(r0 + e) * D + jj];
            } else {
              bfg = sF[r0 * D + jj];
            }
            acc = M::mma(M::load(sdY + c * R2 + r0), bfg, acc);
          }
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            const size_t e = (tokbase + (size_t)t * H) * D + jj;
            dq[e] = (T)(dqv[r] + acc[r]);
            dk[e] = (T)dkv[r];
          }
          if (w == 0 && lane < BLW) {
            float db = sDb2[lane];
            for (int x = 0; x < NW; ++x) db += sDb[x * BLW + lane];
            dbeta[tokbase + (size_t)lane * H] = (T)db;
          }
          for (int rt = 0; rt < R2 / 16; ++rt) {
            if constexpr (sizeof(T) == 2) {
              typename M::frag af, bfg;
              for (int e = 0; e < 4; ++e) {
                af[e] = sdYT[(16 * rt + c) * BLW + 4 * g + e];
                bfg[e] = (T)qv[e];
                af[4 + e] = (T)0.0f;
                bfg[4 + e] = (T)0.0f;
              }
              dF[rt] = M::mma(af, bfg, dF[rt]);
            } else {
              for (int r = 0; r < 4; ++r) dF[rt] = M::mma(sdYT[(16 * rt + c) * BLW + 4 * g + r], qv[r], dF[rt]);
            }
          }
          for (int it = 0; it < NIT; ++it) {
            f32x4 acc1, acc2;
            for (int r = 0; r < 4; ++r) acc1[r] = dS[it][r] * gam;
            acc1 = mma_k16<T>(acc1, sdOT + (16 * it + c) * BLW, sQT + (16 * w + c) * BLW, g);
            acc2 = mma_k16<T>(zero4(), sdET + (16 * it + c) * BLW, sKT + (16 * w + c) * BLW, g);
            for (int r = 0; r < 4; ++r) dS[it][r] = acc1[r] - acc2[r];
          }
        }
      }  // tiles
    }    // passes

    // ---- chunk start: glue through the folded read-out ------------------------
    __syncthreads();
    for (int rt = 0; rt < R2 / 16; ++rt) store_tile(sdF, D, 16 * rt, 16 * w, dF[rt], lane);
    // dS += [Ub;Uw]^T dF  (contraction over the rows of dF, held in registers)
    for (int it = 0; it < NIT; ++it) {
      f32x4 acc = dS[it];
      const int ii = 16 * it + c;  // value row this lane supplies as A
      if constexpr (KPL == 8) {
        for (int ks = 0; ks < R2 / 32; ++ks) {
          typename M::frag af, bfg;
          for (int e = 0; e < 8; ++e) {
            const int rr = 32 * ks + (e < 4 ? 4 * g + e : 16 + 4 * g + e - 4);
            float uv = 0.0f;
            if (rr < R) uv = a.Ub[(size_t)rr * D + ii];
            else if (rr >= RP && rr < RP + R) uv = a.Uw[(size_t)(rr - RP) * D + ii];
            af[e] = (T)uv;
            bfg[e] = (T)(e < 4 ? dF[2 * ks][e] : dF[2 * ks + 1][e - 4]);
          }
          acc = M::mma(af, bfg, acc);
        }
      } else {
        for (int rt = 0; rt < R2 / 16; ++rt)
          for (int r4 = 0; r4 < 4; ++r4) {
            const int rr = 16 * rt + 4 * g + r4;
            float uv = 0.0f;
            if (rr < R) uv = a.Ub[(size_t)rr * D + ii];
            else if (rr >= RP && rr < RP + R) uv = a.Uw[(size_t)(rr - RP) * D + ii];
            acc = M::mma(uv, dF[rt][r4], acc);
          }
      }
      dS[it] = acc;
    }
    __syncthreads();
    // d[Ub;Uw] += dF S_hat^T  (sS still holds S_hat from the first tile)
    for (int rt = 0; rt < R2 / 16; ++rt) {
      f32x4 acc = zero4();
      for (int ks = 0; ks < D / KS; ++ks) {
        const int kofs = ks * KS + g * KPL;
        acc = M::mma(M::load(sdF + (16 * rt + c) * D + kofs), M::load(sS + (16 * w + c) * D + kofs), acc);
      }
      for (int r = 0; r < 4; ++r) {
        const int rr = 16 * rt + 4 * g + r;
        if (rr < R) pUb[(size_t)rr * D + jj] += acc[r];
        else if (rr >= RP && rr < RP + R) pUw[(size_t)(rr - RP) * D + jj] += acc[r];
      }
    }
  }  // chunks

  if (a.dS0) {
    for (int it = 0; it < NIT; ++it)
      for (int r = 0; r < 4; ++r) a.dS0[soff + (size_t)(16 * it + 4 * g + r) * D + jj] = dS[it][r];
  }
  for (int rt = 0; rt < RP / 16; ++rt)
    for (int r = 0; r < 4; ++r) {
      const int j = 16 * w + 4 * g + r, col = 16 * rt + c;
      if (col < R) {
        pVb[(size_t)j * R + col] = dVb[rt][r];
        pVw[(size_t)j * R + col] = dVw[rt][r];
      }
    }
}

// Sum the per-(batch, head) partial parameter gradients in a fixed order.
__global__ void carve_param_reduce_kernel(const float* __restrict__ part, int nparts, size_t rec,
                                          float* dUb, float* dUw, float* dVb, float* dVw, size_t RD) {
  const size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= rec) return;
  float s = 0.0f;
  for (int p = 0; p < nparts; ++p) s += part[(size_t)p * rec + x];
  const size_t which = x / RD, off = x % RD;
  float* dst = which == 0 ? dUb : which == 1 ? dUw : which == 2 ? dVb : dVw;
  dst[off] = s;
}

// ---------------------------------------------------------------------------
template <typename T, int D>
static int launch_bwd_t(const BwdArgs& a, hipStream_t stream) {
  const BwdLds lay = bwd_lds<T, D>(a.RP);
  auto kern = carve_bwd_kernel<T, D>;
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lay.total) != hipSuccess)
      return CARVE_ERR_HIP;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(a.B * a.H), dim3(D * 4), lay.total, stream, a);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

int launch_bwd(const BwdArgs& a, int dtype, int D, int LW, hipStream_t s) {
  if (LW != BLW) return CARVE_ERR_UNSUPPORTED;
  if (dtype == CARVE_BF16) {
    if (D == 32) return launch_bwd_t<bf16_t, 32>(a, s);
    if (D == 64) return launch_bwd_t<bf16_t, 64>(a, s);
    if (D == 128) return launch_bwd_t<bf16_t, 128>(a, s);
  } else {
    if (D == 32) return launch_bwd_t<float, 32>(a, s);
    if (D == 64) return launch_bwd_t<float, 64>(a, s);
  }
  return CARVE_ERR_UNSUPPORTED;
}

size_t bwd_lds_bytes(int dtype, int D, int LW, int RP) {
  if (LW != BLW) return (size_t)-1;
  if (dtype == CARVE_BF16) {
    if (D == 32) return bwd_lds<bf16_t, 32>(RP).total;
    if (D == 64) return bwd_lds<bf16_t, 64>(RP).total;
    if (D == 128) return bwd_lds<bf16_t, 128>(RP).total;
  } else {
    if (D == 32) return bwd_lds<float, 32>(RP).total;
    if (D == 64) return bwd_lds<float, 64>(RP).total;
  }
  return (size_t)-1;
}

int launch_param_reduce(const float* part, int nparts, int R, int D, float* dUb, float* dUw,
                        float* dVb, float* dVw, hipStream_t s) {
  const size_t rec = part_floats(R, D);
  const size_t RD = (size_t)R * D;
  const int threads = 256;
  const int blocks = (int)((rec + threads - 1) / threads);
  hipLaunchKernelGGL(carve_param_reduce_kernel, dim3(blocks), dim3(threads), 0, s, part, nparts, rec, dUb,
                     dUw, dVb, dVw, RD);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

}  // namespace carve
