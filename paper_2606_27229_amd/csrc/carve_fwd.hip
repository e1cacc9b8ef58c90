// carve_fwd.hip -- chunked CARVE forward on gfx950.
//
// One workgroup per (batch, head) runs the whole sequence as a persistent
// loop over gate chunks of L tokens (Alg. carve_fwd).  The recurrent state
// S (Dv x Dk, f32) stays in registers for the whole call: wave w owns the key
// column tiles [w*CPW, (w+1)*CPW) of S (16 columns each) for every value row,
// in the MFMA result layout.  The shared parameters are staged in LDS once,
// and the token inputs of the next WY tile are fetched into registers while
// the current tile computes.
//
// Per gate chunk c (state S_hat = S at the chunk start, Eq. content_readout):
//   F = [Ub; Uw] S_hat            fold, read straight from the S registers
// and then per WY tile of LW <= L tokens (the WY form of Sec. 6.2 applied to
// consecutive sub-blocks of the chunk; the gates of every sub-block use the
// same F, so this is the same computation as one L-token solve):
//   tau = tanh(Q F^T), z_b = bx + tau_b Vb^T, z_w = wx + tau_w Vw^T
//   l = g - softplus(z_b) (log of exp(g)(1-b)), w = sigmoid(z_w)
//   Lam = prefix sums of l inside the tile, handled per 16-token block:
//     E_t = e^{Lam_t - base}, E'_t = e^{Lam_{t-1} - base}, Kinv_t = k_t e^{base - Lam_t}
//     with base = Lam at the end of the previous 16-block.
//   A_ts = beta_t sum_j k_t k_s e^{Lam_{t-1}-Lam_s}   (s < t), built per 16x16
//          tile as (k*E')_t . (Kinv_s * e^{base_ti - base_si}) so that no factor
//          exceeds e^{(16-token log retention)} (Eq. M_coupling, re-derived)
//   P_ts = sum_j q_t k_s e^{Lam_t - Lam_s}              (s <= t), same tiles
//   T = (I + A)^{-1}   16x16 diagonal blocks by forward substitution, the
//                      off-diagonal blocks by block substitution on MFMA
//   R = beta (w*v - Ktil S^T), Ktil_t = k_t e^{Lam_{t-1}};  u = T R
//   O = Qtil S^T + P u, Qtil_t = q_t e^{Lam_t}
//   S <- S diag(e^{Lam_{LW-1}}) + u^T Khat, Khat_s = k_s e^{Lam_{LW-1} - Lam_s}
//
// Precondition (not checked): within any 16-token block the log retention
// summed over the block stays above about -80 per key channel, so that
// e^{-(block log retention)} is finite in f32.
#include "carve_kernels.h"

namespace carve {

template <typename T, int D, int LW>
__global__ void __launch_bounds__(fwd_threads(D)) carve_fwd_kernel(FwdArgs a) {
  typedef Mma<T> M;
  constexpr int NT = fwd_threads(D);
  constexpr int NW = NT / 64;         // waves
  constexpr int NCT = D / 16;         // 16-column tiles of S (key side) / of the value side
  constexpr int CPW = NCT / NW;       // column tiles per wave
  constexpr int NB = LW / 16;         // 16-token blocks per WY tile
  constexpr int NIT = D / 16;         // value-row tiles
  constexpr int KS = M::KS, KPL = M::KPL;
  constexpr int LK = lk_of<T, LW>();  // padded token extent of the K = LW products
  // LDS row strides: every row is padded by 16 bytes so that the 16 rows read by
  // one MFMA fragment load fall into distinct banks
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDD = D + PAD;        // rows of D elements
  constexpr int LDK = LK + PAD;       // rows of LK elements
  constexpr int LDA = LW + 4;         // rows of the f32 coupling matrix
  constexpr int VEC = 16 / sizeof(T); // elements per 16-byte vector
  constexpr int NVT = LW * D / VEC;                // 16-byte vectors of a q (or k) tile
  constexpr int NQV = (NVT + NT - 1) / NT;         // per thread
  const int RP = a.RP, R2 = 2 * a.RP, R = a.R;
  const int LDR = R2 + PAD, LDV = RP + PAD;  // rows of 2RP / RP elements
  const int H = a.H, Tn = a.T, L = a.L;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int nch = Tn / L, msub = L / LW, ntiles = Tn / LW;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const FwdLds lay = fwd_lds<T, D, LW>(RP);
  T* sS = reinterpret_cast<T*>(smem + lay.S);
  T* sQ = reinterpret_cast<T*>(smem + lay.Q);
  T* sK = reinterpret_cast<T*>(smem + lay.K);
  T* sKi = reinterpret_cast<T*>(smem + lay.Ki);
  T* sF = reinterpret_cast<T*>(smem + lay.F);
  T* sTau = reinterpret_cast<T*>(smem + lay.Tau);
  T* sTb = sTau;                                  // alias: T, after tau is dead
  T* sKhT = reinterpret_cast<T*>(smem + lay.KhT);
  float* sA = reinterpret_cast<float*>(smem + lay.A);
  T* sRT = sQ;                                    // alias: R^T [D][LK]
  T* sUT = sK;                                    // alias: u^T [D][LK]
  T* sP = sKi;                                    // alias: P [LW][LK]
  float* sBase = reinterpret_cast<float*>(smem + lay.Base);   // [NB][D]  e^{base_ti}
  float* sCf = reinterpret_cast<float*>(smem + lay.Cf);       // [NB*NB][D] e^{base_ti - base_si}
  float* sBeta = reinterpret_cast<float*>(smem + lay.Beta);   // [LW]
  T* sU = reinterpret_cast<T*>(smem + lay.Ucat);              // [2RP][D] padded [Ub; Uw]
  T* sVb = reinterpret_cast<T*>(smem + lay.Vb);               // [D][RP]
  T* sVw = reinterpret_cast<T*>(smem + lay.Vw);               // [D][RP]

  const T* __restrict__ q = reinterpret_cast<const T*>(a.q);
  const T* __restrict__ k = reinterpret_cast<const T*>(a.k);
  const T* __restrict__ v = reinterpret_cast<const T*>(a.v);
  const T* __restrict__ bx = reinterpret_cast<const T*>(a.bx);
  const T* __restrict__ wx = reinterpret_cast<const T*>(a.wx);
  const T* __restrict__ beta = reinterpret_cast<const T*>(a.beta);
  // token tensors addressed from this (batch, head)'s first element with 32-bit
  // offsets t * rs + column (rs = H * D elements between consecutive tokens)
  const size_t bh0 = ((size_t)b * Tn * H + h) * D;
  const size_t bh1 = (size_t)b * Tn * H + h;
  const int rs = H * D;
  q += bh0; k += bh0; v += bh0; bx += bh0; wx += bh0; beta += bh1;
  const float* __restrict__ gl = a.g + bh0;
  T* __restrict__ o = reinterpret_cast<T*>(a.o) + bh0;

  // ---- shared parameters -> LDS (zero padded to RP) ------------------------
  for (int x = tid; x < R2 * D; x += NT) {
    const int rr = x / D, i = x % D;
    float u = 0.0f;
    if (rr < R) u = a.Ub[(size_t)rr * D + i];
    else if (rr >= RP && rr < RP + R) u = a.Uw[(size_t)(rr - RP) * D + i];
    sU[rr * LDD + i] = (T)u;
  }
  for (int x = tid; x < D * RP; x += NT) {
    const int j = x / RP, rr = x % RP;
    sVb[j * LDV + rr] = (T)(rr < R ? a.Vb[(size_t)j * R + rr] : 0.0f);
    sVw[j * LDV + rr] = (T)(rr < R ? a.Vw[(size_t)j * R + rr] : 0.0f);
  }

  // ---- state registers: S[cq][it][r] = S[16*it + 4g + r][16*(w*CPW+cq) + c] ----
  f32x4 S[CPW][NIT];
  const size_t soff = (size_t)bh * D * D;
  for (int cq = 0; cq < CPW; ++cq) {
    const int col = 16 * (w * CPW + cq) + c;
    for (int it = 0; it < NIT; ++it) {
      for (int r = 0; r < 4; ++r)
        S[cq][it][r] = a.S0 ? a.S0[soff + (size_t)(16 * it + 4 * g + r) * D + col] : 0.0f;
      store_tile(sS, LDD, 16 * it, 16 * (w * CPW + cq), S[cq][it], lane);
    }
  }

  // ---- prefetch registers for the next WY tile ---------------------------
  f32x4 pq[NQV], pk[NQV];
  float pbx[CPW][NB][4], pg[CPW][NB][4], pwx[CPW][NB][4], pv[CPW][NB][4];
  float pbeta = 0.0f;
#define CARVE_FWD_PREFETCH_QK(TILE_)                                                    \
  do {                                                                                  \
    const int tt0_ = (TILE_) * LW;                                                      \
    for (int u = 0; u < NQV; ++u) {                                                     \
      const int x = tid + u * NT;                                                       \
      if (NVT % NT != 0 && x >= NVT) break;                                             \
      const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;                           \
      const int gofs = (tt0_ + t) * rs + j;                                             \
      pq[u] = *reinterpret_cast<const f32x4*>(q + gofs);                                \
      pk[u] = *reinterpret_cast<const f32x4*>(k + gofs);                                \
    }                                                                                   \
    if (tid < LW) pbeta = to_f(beta[(tt0_ + tid) * H]);                                 \
  } while (0)
#define CARVE_FWD_PREFETCH_GATES(TILE_)                                                 \
  do {                                                                                  \
    const int tt0_ = (TILE_) * LW;                                                      \
    for (int cq = 0; cq < CPW; ++cq) {                                                  \
      const int col_ = 16 * (w * CPW + cq) + c;                                         \
      for (int ti = 0; ti < NB; ++ti)                                                   \
        for (int r = 0; r < 4; ++r) {                                                   \
          const int e_ = (tt0_ + 16 * ti + 4 * g + r) * rs + col_;                      \
          pbx[cq][ti][r] = to_f(bx[e_]);                                                \
          pg[cq][ti][r] = gl[e_];                                                       \
          pwx[cq][ti][r] = to_f(wx[e_]);                                                \
          pv[cq][ti][r] = to_f(v[e_]);                                                  \
        }                                                                               \
    }                                                                                   \
  } while (0)
  CARVE_FWD_PREFETCH_QK(0);
  CARVE_FWD_PREFETCH_GATES(0);

  for (int ch = 0; ch < nch; ++ch) {
    if (a.S_chunks) {
      float* dst = a.S_chunks + ((size_t)bh * nch + ch) * D * D;
      for (int cq = 0; cq < CPW; ++cq) {
        const int col = 16 * (w * CPW + cq) + c;
        for (int it = 0; it < NIT; ++it)
          for (int r = 0; r < 4; ++r) dst[(size_t)(16 * it + 4 * g + r) * D + col] = S[cq][it][r];
      }
    }
    for (int m = 0; m < msub; ++m) {
      const int tile = ch * msub + m;
      const int t0 = tile * LW;

      // ---- P0: q, k tiles and beta from the prefetch registers -------------
      for (int u = 0; u < NQV; ++u) {
        const int x = tid + u * NT;
        if (NVT % NT != 0 && x >= NVT) break;
        const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;
        *reinterpret_cast<f32x4*>(sQ + t * LDD + j) = pq[u];
        *reinterpret_cast<f32x4*>(sK + t * LDD + j) = pk[u];
      }
      if (tid < LW) sBeta[tid] = pbeta;
      if (tile + 1 < ntiles) CARVE_FWD_PREFETCH_QK(tile + 1);
      // ---- P1: fold F = [Ub;Uw] S_hat from the state registers ---------------
      if (m == 0) {
        for (int cq = 0; cq < CPW; ++cq) {
          const int ct = w * CPW + cq;
          for (int rt = 0; rt < R2 / 16; ++rt) {
            const T* urow = sU + (16 * rt + c) * LDD;  // B row this lane supplies
            f32x4 acc = zero4();
            if constexpr (KPL == 8) {
              for (int ks = 0; ks < D / 32; ++ks) {
                typename M::frag af, bfg;
                const T* p = urow + 32 * ks + 4 * g;
                for (int e = 0; e < 4; ++e) {
                  af[e] = (T)S[cq][2 * ks][e];
                  af[4 + e] = (T)S[cq][2 * ks + 1][e];
                  bfg[e] = p[e];
                  bfg[4 + e] = p[16 + e];
                }
                acc = M::mma(af, bfg, acc);
              }
            } else {
              for (int it = 0; it < NIT; ++it)
                for (int r4 = 0; r4 < 4; ++r4) acc = M::mma((T)S[cq][it][r4], urow[16 * it + 4 * g + r4], acc);
            }
            // acc = F^T[j = 16ct + 4g + r][16rt + c]  ->  sF[r][j]
            store_tile_t(sF, LDD, 16 * ct, 16 * rt, acc, lane);
          }
        }
      }
      __syncthreads();

      // ---- P2: tau = tanh(Q F^T) -> sTau [LW][2RP] ----------------------------
      {
        const int ntl = NB * (R2 / 16);
        for (int x = w; x < ntl; x += NW) {
          const int ti = x / (R2 / 16), rt = x % (R2 / 16);
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sQ + (16 * ti + c) * LDD + kofs), M::load(sF + (16 * rt + c) * LDD + kofs), acc);
          }
          for (int r = 0; r < 4; ++r) acc[r] = tanh_f(acc[r]);
          store_tile(sTau, LDR, 16 * ti, 16 * rt, acc, lane);
        }
      }
      __syncthreads();

      // ---- P3: gate logits (key side: l; value side: w*v) --------------------
      float ell[CPW][NB][4];
      float wv[CPW][NB][4];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const T* vbrow = sVb + (16 * ct + c) * LDV;
        const T* vwrow = sVw + (16 * ct + c) * LDV;
        for (int ti = 0; ti < NB; ++ti) {
          f32x4 accB = zero4(), accW = zero4();
          for (int ks = 0; ks < RP / KS; ++ks) {
            const int r0 = ks * KS + g * KPL;
            const int arow = (16 * ti + c) * LDR;
            accB = M::mma(M::load(sTau + arow + r0), M::load(vbrow + r0), accB);
            accW = M::mma(M::load(sTau + arow + RP + r0), M::load(vwrow + r0), accW);
          }
          for (int r = 0; r < 4; ++r) {
            const float zb = pbx[cq][ti][r] + accB[r];
            ell[cq][ti][r] = pg[cq][ti][r] - softplus_f(zb);
            wv[cq][ti][r] = sigmoid_f(pwx[cq][ti][r] + accW[r]) * pv[cq][ti][r];
          }
        }
      }
      if (tile + 1 < ntiles) CARVE_FWD_PREFETCH_GATES(tile + 1);

      // ---- P4: key-side retention factors --------------------------------------
      float gamma_col[CPW];  // e^{Lam_{LW-1}} for key column 16(w*CPW+cq) + c
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        float base = 0.0f;  // Lam at the end of the previous block
        float bases[NB];
        for (int ti = 0; ti < NB; ++ti) {
          float p[4];
          p[0] = ell[cq][ti][0];
          p[1] = p[0] + ell[cq][ti][1];
          p[2] = p[1] + ell[cq][ti][2];
          p[3] = p[2] + ell[cq][ti][3];
          float incl = p[3];
          float y = __shfl_up(incl, 16);
          if (g >= 1) incl += y;
          y = __shfl_up(incl, 32);
          if (g >= 2) incl += y;
          const float excl = incl - p[3];
          const float btot = __shfl(incl, 48 + c);   // block log retention
          float E[4], Ep[4], Ki[4];
          for (int r = 0; r < 4; ++r) {
            const float lrel = excl + p[r];
            E[r] = fast_exp(lrel);
            Ki[r] = fast_exp(-lrel);
          }
          const float Eprev = __shfl_up(E[3], 16);
          Ep[0] = g == 0 ? 1.0f : Eprev;
          Ep[1] = E[0];
          Ep[2] = E[1];
          Ep[3] = E[2];
          for (int r = 0; r < 4; ++r) {
            const int t = 16 * ti + 4 * g + r;
            const float kv = to_f(sK[t * LDD + jj]);
            const float qv = to_f(sQ[t * LDD + jj]);
            sK[t * LDD + jj] = (T)(kv * Ep[r]);
            sQ[t * LDD + jj] = (T)(qv * E[r]);
            Ki[r] *= kv;
            sKi[t * LDD + jj] = (T)Ki[r];
            ell[cq][ti][r] = Ki[r];  // keep k e^{-Lam_rel}
          }
          bases[ti] = base;
          base += btot;
        }
        const float lam_end = base;  // Lam_{LW-1}
        gamma_col[cq] = fast_exp(lam_end);
        for (int ti = 0; ti < NB; ++ti) {
          // Khat^T[j][s] = Kinv_s e^{Lam_end - base_si}
          const float f = fast_exp(lam_end - bases[ti]);
          f32x4 kh;
          for (int r = 0; r < 4; ++r) kh[r] = ell[cq][ti][r] * f;
          store_tile_t(sKhT, LDK, 16 * ti, 16 * ct, kh, lane);
          if (g == 0) {
            sBase[ti * D + jj] = fast_exp(bases[ti]);
            for (int si = 0; si < ti; ++si) sCf[(ti * NB + si) * D + jj] = fast_exp(bases[ti] - bases[si]);
          }
        }
      }
      __syncthreads();

      // ---- P5: A, P (lower 16x16 tiles) and Ktil S^T, Qtil S^T ------------------
      constexpr int NTRI = NB * (NB + 1) / 2;
      constexpr int PPW = (NTRI + NW - 1) / NW;
      f32x4 Pkeep[PPW];
      {
        int slot = 0;
        for (int x = w; x < NTRI; x += NW, ++slot) {
          int ti = 0, si = x;
          while (si > ti) { si -= ti + 1; ++ti; }
          f32x4 accA = zero4(), accP = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            const T* kb = sKi + (16 * si + c) * LDD + kofs;
            const typename M::frag bf = (ti == si) ? M::load(kb) : M::load_scaled(kb, sCf + (ti * NB + si) * D + kofs);
            accA = M::mma(M::load(sK + (16 * ti + c) * LDD + kofs), bf, accA);
            accP = M::mma(M::load(sQ + (16 * ti + c) * LDD + kofs), bf, accP);
          }
          for (int r = 0; r < 4; ++r) {
            const int tl = 4 * g + r;  // row inside the tile
            const bool lowA = (ti > si) || (c < tl);
            const bool lowP = (ti > si) || (c <= tl);
            sA[(16 * ti + tl) * LDA + 16 * si + c] = lowA ? sBeta[16 * ti + tl] * accA[r] : 0.0f;
            accP[r] = lowP ? accP[r] : 0.0f;
          }
          Pkeep[slot] = accP;
        }
      }
      f32x4 XK[CPW][NB], XQ[CPW][NB];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        for (int ti = 0; ti < NB; ++ti) {
          f32x4 ak = zero4(), aq = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            const typename M::frag sb = M::load(sS + (16 * ct + c) * LDD + kofs);
            const float* sc = sBase + ti * D + kofs;
            ak = M::mma(M::load_scaled(sK + (16 * ti + c) * LDD + kofs, sc), sb, ak);
            aq = M::mma(M::load_scaled(sQ + (16 * ti + c) * LDD + kofs, sc), sb, aq);
          }
          XK[cq][ti] = ak;
          XQ[cq][ti] = aq;
        }
      }
      __syncthreads();
      // epilogues into the aliased buffers
      {
        int slot = 0;
        for (int x = w; x < NTRI; x += NW, ++slot) {
          int ti = 0, si = x;
          while (si > ti) { si -= ti + 1; ++ti; }
          store_tile(sP, LDK, 16 * ti, 16 * si, Pkeep[slot], lane);
        }
        // zero the upper tiles (and padding columns) of P and T, and the
        // padding columns of R^T, u^T and Khat^T (read by the 32-wide K steps)
        for (int x = tid; x < LW * LK; x += NT) {
          const int rr = x / LK, cc = x % LK;
          if ((cc >> 4) > (rr >> 4)) {
            sP[rr * LDK + cc] = (T)0.0f;
            sTb[rr * LDK + cc] = (T)0.0f;
          }
        }
        if constexpr (LK > LW) {
          for (int x = tid; x < D * (LK - LW); x += NT) {
            const int rr = x / (LK - LW), cc = LW + x % (LK - LW);
            sRT[rr * LDK + cc] = (T)0.0f;
            sUT[rr * LDK + cc] = (T)0.0f;
            sKhT[rr * LDK + cc] = (T)0.0f;
          }
        }
        for (int cq = 0; cq < CPW; ++cq)
          for (int ti = 0; ti < NB; ++ti) {
            f32x4 rv;
            for (int r = 0; r < 4; ++r) rv[r] = sBeta[16 * ti + 4 * g + r] * (wv[cq][ti][r] - XK[cq][ti][r]);
            store_tile_t(sRT, LDK, 16 * ti, 16 * (w * CPW + cq), rv, lane);
          }
      }
      __syncthreads();

      // ---- P6: T = (I + A)^{-1} -----------------------------------------------
      if (w == 0 && g < NB) {
        // diagonal block g: column c by forward substitution, A rows in registers
        const float* Ab = sA + (16 * g) * LDA + 16 * g;
        float arow[16][16];
#pragma unroll
        for (int t = 1; t < 16; ++t)
#pragma unroll
          for (int s4 = 0; s4 < (t + 3) / 4; ++s4) {
            const f32x4 v4 = *reinterpret_cast<const f32x4*>(Ab + t * LDA + 4 * s4);
            arow[t][4 * s4] = v4[0];
            arow[t][4 * s4 + 1] = v4[1];
            arow[t][4 * s4 + 2] = v4[2];
            arow[t][4 * s4 + 3] = v4[3];
          }
        float x[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          float acc = (t == c) ? 1.0f : 0.0f;
#pragma unroll
          for (int s = 0; s < t; ++s) acc -= arow[t][s] * x[s];
          x[t] = acc;
        }
        float* Aw = sA + (16 * g) * LDA + 16 * g;
        T* Tw = sTb + (16 * g) * LDK + 16 * g;
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          Aw[t * LDA + c] = x[t];
          Tw[t * LDK + c] = (T)x[t];
        }
      }
      __syncthreads();
      if constexpr (NB > 1) {
        for (int j = w; j < NB - 1; j += NW) {
          f32x4 Tc[NB];
          for (int i = j + 1; i < NB; ++i) {
            f32x4 X = zero4();
            for (int kb = j; kb < i; ++kb) {
              for (int ks = 0; ks < 4; ++ks) {
                const float av = sA[(16 * i + c) * LDA + 16 * kb + 4 * g + ks];
                const float bv = (kb == j) ? sA[(16 * kb + 4 * g + ks) * LDA + 16 * j + c] : Tc[kb][ks];
                X = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, X, 0, 0, 0);
              }
            }
            f32x4 Y = zero4();
            for (int ks = 0; ks < 4; ++ks) {
              const float av = sA[(16 * i + c) * LDA + 16 * i + 4 * g + ks];
              Y = __builtin_amdgcn_mfma_f32_16x16x4f32(av, X[ks], Y, 0, 0, 0);
            }
            for (int r = 0; r < 4; ++r) Y[r] = -Y[r];
            Tc[i] = Y;
            store_tile(sTb, LDK, 16 * i, 16 * j, Y, lane);
          }
        }
        __syncthreads();
      }

      // ---- P7: u = T R -> sUT -----------------------------------------------
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        for (int ti = 0; ti < NB; ++ti) {
          f32x4 acc = zero4();
          const int kmax = (16 * (ti + 1) + KS - 1) / KS;
          for (int ks = 0; ks < kmax; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sTb + (16 * ti + c) * LDK + kofs), M::load(sRT + (16 * ct + c) * LDK + kofs), acc);
          }
          store_tile_t(sUT, LDK, 16 * ti, 16 * ct, acc, lane);
        }
      }
      __syncthreads();

      // ---- P8: outputs and state carry --------------------------------------
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        for (int ti = 0; ti < NB; ++ti) {
          f32x4 acc = XQ[cq][ti];
          const int kmax = (16 * (ti + 1) + KS - 1) / KS;
          for (int ks = 0; ks < kmax; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sP + (16 * ti + c) * LDK + kofs), M::load(sUT + (16 * ct + c) * LDK + kofs), acc);
          }
          for (int r = 0; r < 4; ++r) {
            const int t = 16 * ti + 4 * g + r;
            o[(t0 + t) * rs + 16 * ct + c] = (T)acc[r];
          }
        }
      }
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        for (int it = 0; it < NIT; ++it) {
          f32x4 acc;
          for (int r = 0; r < 4; ++r) acc[r] = S[cq][it][r] * gamma_col[cq];
          for (int ks = 0; ks < LK / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load(sUT + (16 * it + c) * LDK + kofs), M::load(sKhT + (16 * ct + c) * LDK + kofs), acc);
          }
          S[cq][it] = acc;
        }
      }
      __syncthreads();  // every wave is done reading sS (P5) and the aliases
      for (int cq = 0; cq < CPW; ++cq)
        for (int it = 0; it < NIT; ++it) store_tile(sS, LDD, 16 * it, 16 * (w * CPW + cq), S[cq][it], lane);
    }
  }
  if (a.S_T) {
    for (int cq = 0; cq < CPW; ++cq) {
      const int col = 16 * (w * CPW + cq) + c;
      for (int it = 0; it < NIT; ++it)
        for (int r = 0; r < 4; ++r) a.S_T[soff + (size_t)(16 * it + 4 * g + r) * D + col] = S[cq][it][r];
    }
  }
}

// ---------------------------------------------------------------------------
// host-side launch
// ---------------------------------------------------------------------------
template <typename T, int D, int LW>
static int launch_fwd_t(const FwdArgs& a, hipStream_t stream) {
  const FwdLds lay = fwd_lds<T, D, LW>(a.RP);
  auto kern = carve_fwd_kernel<T, D, LW>;
  static bool attr_set = false;  // per instantiation
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lay.total) != hipSuccess)
      return CARVE_ERR_HIP;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(a.B * a.H), dim3(fwd_threads(D)), lay.total, stream, a);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T>
static int launch_fwd_d(const FwdArgs& a, int D, int LW, hipStream_t s) {
#define CARVE_FWD_CASE(DD, LL) \
  if (D == DD && LW == LL) return launch_fwd_t<T, DD, LL>(a, s);
  CARVE_FWD_CASE(32, 16) CARVE_FWD_CASE(32, 32) CARVE_FWD_CASE(32, 64)
  CARVE_FWD_CASE(64, 16) CARVE_FWD_CASE(64, 32) CARVE_FWD_CASE(64, 64)
  CARVE_FWD_CASE(128, 16) CARVE_FWD_CASE(128, 32) CARVE_FWD_CASE(128, 64)
#undef CARVE_FWD_CASE
  return CARVE_ERR_UNSUPPORTED;
}

int launch_fwd(const FwdArgs& a, int dtype, int D, int LW, hipStream_t s) {
  if (dtype == CARVE_BF16) return launch_fwd_d<bf16_t>(a, D, LW, s);
  return launch_fwd_d<float>(a, D, LW, s);
}

size_t fwd_lds_bytes(int dtype, int D, int LW, int RP) {
#define CARVE_LDS_CASE(DD, LL)                                                              \
  if (D == DD && LW == LL)                                                                  \
    return dtype == CARVE_BF16 ? fwd_lds<bf16_t, DD, LL>(RP).total : fwd_lds<float, DD, LL>(RP).total;
  CARVE_LDS_CASE(32, 16) CARVE_LDS_CASE(32, 32) CARVE_LDS_CASE(32, 64)
  CARVE_LDS_CASE(64, 16) CARVE_LDS_CASE(64, 32) CARVE_LDS_CASE(64, 64)
  CARVE_LDS_CASE(128, 16) CARVE_LDS_CASE(128, 32) CARVE_LDS_CASE(128, 64)
#undef CARVE_LDS_CASE
  return (size_t)-1;
}

}  // namespace carve
