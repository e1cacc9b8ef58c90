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

// Compiler-only fence: keeps the loads of one unrolled iteration from being
// hoisted above the previous one (bounds the live fragment registers).
#define CARVE_SEQ() asm volatile("" ::: "memory")

struct BwdLds {
  size_t S, dS, F, Q, K, Ki, QT, KT, KiT, Tau, A, Dm, Tb, TbT, PT, RT, U, UTz, KhTz, dO, dOT, duT,
      dET, Gam, Beta, Db, Db2, total;
};

template <typename T, int D>
__host__ __device__ constexpr BwdLds bwd_lds(int RP) {
  BwdLds l{};
  size_t off = 0;
  const size_t e = sizeof(T);
  constexpr size_t PAD = 16 / sizeof(T);        // every LDS row is padded by 16 bytes
  constexpr size_t LDD = D + PAD, LDB = BLW, LDF = BLW + 4;
  const size_t R2 = 2 * (size_t)RP, LDR = R2 + PAD;
  constexpr size_t RD = (size_t)BLW * LDD;   // [16][D]
  constexpr size_t DR = (size_t)D * LDB;     // [D][16]
  constexpr size_t LL = (size_t)BLW * LDB;   // [16][16]
  constexpr size_t LLF = (size_t)BLW * LDF;  // [16][16] f32
  l.S = off;    off += lds_round((size_t)D * LDD * e);
  l.dS = off;   off += lds_round((size_t)D * LDD * e);
  l.F = off;    off += lds_round(R2 * LDD * e);
  // transient region; dF (R2 x D) for the parameter product at a chunk start
  // reuses it once the tiles of the chunk are done
  l.Q = off;    off += lds_round(RD * e);
  l.K = off;    off += lds_round(RD * e);
  l.Ki = off;   off += lds_round(RD * e);
  l.QT = off;   off += lds_round(DR * e);
  l.KT = off;   off += lds_round(DR * e);
  l.KiT = off;  off += lds_round(DR * e);
  l.Tau = off;  off += lds_round((size_t)BLW * LDR * e);
  l.A = off;    off += lds_round(LLF * 4);
  l.Dm = off;   off += lds_round(LLF * 4);
  l.Tb = off;   off += lds_round(LL * e);
  l.TbT = off;  off += lds_round(LL * e);
  l.PT = off;   off += lds_round(LL * e);
  l.RT = off;   off += lds_max(lds_round(DR * e), lds_round((size_t)BLW * LDR * e) + lds_round(R2 * LDB * e));
  l.U = off;    off += lds_round(RD * e);
  l.UTz = off;  off += lds_round(lds_max(DR, RD) * e);   // u^T (forward tiles) / dz_b (backward tiles)
  l.KhTz = off; off += lds_round(lds_max(DR, RD) * e);   // Khat^T (forward tiles) / dz_w (backward tiles)
  l.dO = off;   off += lds_round(RD * e);
  l.dOT = off;  off += lds_round(DR * e);
  l.duT = off;  off += lds_round(DR * e);
  l.dET = off;  off += lds_round(DR * e);
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

// Column c of (I + A)^{-1} for a 16x16 strictly lower A (row stride lda) by
// forward substitution; the rows of A are read one ahead of their use.
__device__ __forceinline__ void unit_lower_inverse_column(const float* A, int lda, int c, float* x) {
  f32x4 cur[4], nxt[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) cur[s4] = *reinterpret_cast<const f32x4*>(A + 1 * lda + 4 * s4);
  x[0] = (c == 0) ? 1.0f : 0.0f;
#pragma unroll
  for (int t = 1; t < 16; ++t) {
    if (t + 1 < 16) {
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) nxt[s4] = *reinterpret_cast<const f32x4*>(A + (t + 1) * lda + 4 * s4);
    }
    float acc = (t == c) ? 1.0f : 0.0f;
#pragma unroll
    for (int s = 0; s < t; ++s) acc -= cur[s >> 2][s & 3] * x[s];
    x[t] = acc;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) cur[s4] = nxt[s4];
  }
}

// Pack [Ub; Uw] once per call into the workspace, zero padded to RP rows per
// half, in both orientations: Up [2RP][D] and UT [D][2RP] (token dtype).
template <typename T>
__global__ void carve_pack_u_kernel(const float* __restrict__ Ub, const float* __restrict__ Uw, int R, int RP,
                                    int D, T* __restrict__ Up, T* __restrict__ UT) {
  const int x = blockIdx.x * blockDim.x + threadIdx.x;
  const int R2 = 2 * RP;
  if (x >= R2 * D) return;
  const int rr = x / D, i = x % D;
  float u = 0.0f;
  if (rr < R) u = Ub[(size_t)rr * D + i];
  else if (rr >= RP && rr < RP + R) u = Uw[(size_t)(rr - RP) * D + i];
  Up[x] = (T)u;
  UT[(size_t)i * R2 + rr] = (T)u;
}

template <typename T, int D, int RP>
__global__ void __launch_bounds__(bwd_threads(D)) carve_bwd_kernel(BwdArgs a) {
  typedef Mma<T> M;
  constexpr int NT = bwd_threads(D);
  constexpr int NW = NT / 64;
  constexpr int NCT = D / 16;
  constexpr int CPW = NCT / NW;       // column tiles per wave
  constexpr int NIT = D / 16;
  constexpr int KS = M::KS, KPL = M::KPL;
  constexpr int R2 = 2 * RP;
  constexpr int NRT = R2 / 16;        // 16-row tiles of [Ub; Uw]
  constexpr int NVT = RP / 16;        // 16-column tiles of Vb / Vw
  constexpr int VEC = 16 / sizeof(T);
  constexpr int NQV = (BLW * D / VEC + NT - 1) / NT;
  constexpr int NGT = (2 * NVT + NW - 1) / NW;  // dtau tiles per wave
  // LDS row strides, each row padded by 16 bytes so that the 16 rows read by one
  // MFMA fragment load fall into distinct banks
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDD = D + PAD;     // rows of D elements
  constexpr int LDB = BLW;         // rows of 16 tokens (2-way bank conflicts at most)
  constexpr int LDR = R2 + PAD;    // rows of 2RP elements
  constexpr int LDF = BLW + 4;     // rows of the f32 16x16 matrices
  const int R = a.R;
  const int H = a.H, Tn = a.T, L = a.L;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int nch = Tn / L, msub = L / BLW;

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
  T* sdR = sQ;  // alias: Q is dead after R3
  T* sdE = sK;  // alias: K is dead after R3
  T* sdET = reinterpret_cast<T*>(smem + lay.dET);
  // dD, dD^T, dP, dP^T reuse T, T^T, P^T, A (dead after R5); dY, dY^T reuse R^T
  T* sdD = sTb;
  T* sdDT = sTbT;
  T* sdP = sPT;
  T* sdPT = reinterpret_cast<T*>(smem + lay.A);
  T* sdY = sRT;
  T* sdYT = reinterpret_cast<T*>(smem + lay.RT + lds_round((size_t)BLW * LDR * sizeof(T)));
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
  const T* __restrict__ Up = reinterpret_cast<const T*>(a.Up);
  const T* __restrict__ UT = reinterpret_cast<const T*>(a.UT);
  // token tensors addressed from this (batch, head)'s first element with 32-bit
  // offsets t * rs + column (rs = H * D elements between consecutive tokens)
  const size_t bh0 = ((size_t)b * Tn * H + h) * D;
  const size_t bh1 = (size_t)b * Tn * H + h;
  const int rs = H * D;
  q += bh0; k += bh0; v += bh0; bx += bh0; wx += bh0; dO += bh0; beta += bh1;
  const float* __restrict__ gl = a.g + bh0;
  float* __restrict__ dgo = a.dg + bh0;
  T* __restrict__ dq = reinterpret_cast<T*>(a.dq) + bh0;
  T* __restrict__ dk = reinterpret_cast<T*>(a.dk) + bh0;
  T* __restrict__ dv = reinterpret_cast<T*>(a.dv) + bh0;
  T* __restrict__ dbeta = reinterpret_cast<T*>(a.dbeta) + bh1;
  T* __restrict__ dbx = reinterpret_cast<T*>(a.dbx) + bh0;
  T* __restrict__ dwx = reinterpret_cast<T*>(a.dwx) + bh0;
  const size_t soff = (size_t)bh * D * D;

  // ---- constant operand fragments of Vb, Vw -------------------------------------
  // z = x + tau V^T: B[k = r][n = j] = V[j][r]  (per owned column tile, RP/KS steps)
  typename M::frag fVb[CPW][RP / KS], fVw[CPW][RP / KS];
  for (int cq = 0; cq < CPW; ++cq) {
    const int col = 16 * (w * CPW + cq) + c;
    for (int ks = 0; ks < RP / KS; ++ks) {
      float vb[KPL], vw[KPL];
      for (int e = 0; e < KPL; ++e) {
        const int rr = ks * KS + g * KPL + e;
        vb[e] = rr < R ? a.Vb[(size_t)col * R + rr] : 0.0f;
        vw[e] = rr < R ? a.Vw[(size_t)col * R + rr] : 0.0f;
      }
      fVb[cq][ks] = M::from_f32(vb);
      fVw[cq][ks] = M::from_f32(vw);
    }
  }
  // dtau = dz V: B[k = j][n = r] = V[j][r] for the dtau tiles this wave owns
  typename M::frag fVt[NGT][D / KS];
  for (int gi = 0; gi < NGT; ++gi) {
    const int x = w + gi * NW;
    const int half = x / NVT, rt = x % NVT;
    const float* Vm = half ? a.Vw : a.Vb;
    const int col = 16 * rt + c;
    for (int ks = 0; ks < D / KS; ++ks) {
      float vb[KPL];
      for (int e = 0; e < KPL; ++e) {
        const int j = ks * KS + g * KPL + e;
        vb[e] = (x < 2 * NVT && col < R) ? Vm[(size_t)j * R + col] : 0.0f;
      }
      fVt[gi][ks] = M::from_f32(vb);
    }
  }

  // ---- persistent registers --------------------------------------------------------
  // S[cq][it][r] = S[16 it + 4g + r][16(w CPW + cq) + c] (tile start state), dS the
  // gradient of the tile end state, dF the fold gradient of the current chunk,
  // dU / dVb / dVw this (batch, head)'s parameter-gradient partials.
  f32x4 S[CPW][NIT], dS[CPW][NIT], dF[CPW][NRT], dU[CPW][NRT], dVb[CPW][NVT], dVw[CPW][NVT];
  for (int cq = 0; cq < CPW; ++cq) {
    const int col = 16 * (w * CPW + cq) + c;
    for (int it = 0; it < NIT; ++it)
      for (int r = 0; r < 4; ++r) {
        const size_t e = soff + (size_t)(16 * it + 4 * g + r) * D + col;
        dS[cq][it][r] = a.dS_T ? a.dS_T[e] : 0.0f;
        S[cq][it][r] = a.S_chunks[((size_t)bh * nch + nch - 1) * D * D + (16 * it + 4 * g + r) * D + col];
      }
    for (int x = 0; x < NRT; ++x) dU[cq][x] = zero4();
    for (int x = 0; x < NVT; ++x) {
      dVb[cq][x] = zero4();
      dVw[cq][x] = zero4();
    }
  }

  // ---- per-tile input prefetch ----------------------------------------------------
  f32x4 pq[NQV], pk[NQV], pdo[NQV];
  float cbx[CPW][4], cg[CPW][4], cwx[CPW][4], cv[CPW][4];
  float pbeta = 0.0f;
#define CARVE_BWD_PREFETCH_VEC(T0_, WANT_DO_)                                            \
  do {                                                                                   \
    const int t0_ = (T0_);                                                               \
    for (int u = 0; u < NQV; ++u) {                                                      \
      const int x = tid + u * NT;                                                        \
      if ((BLW * D / VEC) % NT != 0 && x >= BLW * D / VEC) break;                        \
      const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;                            \
      const int gofs = (t0_ + t) * rs + j;                                               \
      pq[u] = *reinterpret_cast<const f32x4*>(q + gofs);                                 \
      pk[u] = *reinterpret_cast<const f32x4*>(k + gofs);                                 \
      if (WANT_DO_) pdo[u] = *reinterpret_cast<const f32x4*>(dO + gofs);                 \
    }                                                                                    \
    if (tid < BLW) pbeta = to_f(beta[(t0_ + tid) * H]);                                  \
  } while (0)
#define CARVE_BWD_PREFETCH_GATES(T0_)                                                    \
  do {                                                                                   \
    const int t0_ = (T0_);                                                               \
    for (int cq = 0; cq < CPW; ++cq) {                                                   \
      const int col_ = 16 * (w * CPW + cq) + c;                                          \
      for (int r = 0; r < 4; ++r) {                                                      \
        const int e_ = (t0_ + 4 * g + r) * rs + col_;                                    \
        cbx[cq][r] = to_f(bx[e_]);                                                       \
        cg[cq][r] = gl[e_];                                                              \
        cwx[cq][r] = to_f(wx[e_]);                                                       \
        cv[cq][r] = to_f(v[e_]);                                                         \
      }                                                                                  \
    }                                                                                    \
  } while (0)

  // the tile steps of a chunk: forward tiles 0..msub-2 (recompute the tile start
  // states), then backward tiles msub-1..0
  const int nsteps = 2 * msub - 1;
#define CARVE_STEP_IS_BWD(ST_) ((ST_) >= msub - 1)
#define CARVE_STEP_TILE(ST_) (CARVE_STEP_IS_BWD(ST_) ? (2 * msub - 2 - (ST_)) : (ST_))
  CARVE_BWD_PREFETCH_VEC((nch - 1) * L + CARVE_STEP_TILE(0) * BLW, CARVE_STEP_IS_BWD(0));
  CARVE_BWD_PREFETCH_GATES((nch - 1) * L + CARVE_STEP_TILE(0) * BLW);

  for (int ch = nch - 1; ch >= 0; --ch) {
    for (int cq = 0; cq < CPW; ++cq)
      for (int x = 0; x < NRT; ++x) dF[cq][x] = zero4();
    __syncthreads();
    // ---- fold F = [Ub; Uw] S_hat -> sF [R2][D] (S holds S_hat here) -------------
    for (int cq = 0; cq < CPW; ++cq) {
      const int ct = w * CPW + cq;
      typename M::frag sa[NIT / 2 > 0 ? NIT / 2 : 1];
      if constexpr (KPL == 8)
        for (int ks = 0; ks < NIT / 2; ++ks)
          for (int e = 0; e < 4; ++e) {
            sa[ks][e] = (T)S[cq][2 * ks][e];
            sa[ks][4 + e] = (T)S[cq][2 * ks + 1][e];
          }
      for (int rt = 0; rt < NRT; ++rt) {
        CARVE_SEQ();
        const T* urow = Up + (size_t)(16 * rt + c) * D;
        f32x4 acc = zero4();
        if constexpr (KPL == 8) {
          for (int ks = 0; ks < D / 32; ++ks) {
            typename M::frag bfg;
            const T* p = urow + 32 * ks + 4 * g;
            const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p);
            const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 16);
            for (int e = 0; e < 4; ++e) {
              bfg[e] = lo[e];
              bfg[4 + e] = hi[e];
            }
            acc = M::mma(sa[ks], bfg, acc);
          }
        } else {
          for (int it = 0; it < NIT; ++it)
            for (int r4 = 0; r4 < 4; ++r4) acc = M::mma(S[cq][it][r4], urow[16 * it + 4 * g + r4], acc);
        }
        store_tile_t(sF, LDD, 16 * ct, 16 * rt, acc, lane);
      }
    }

    for (int st = 0; st < nsteps; ++st) {
      const bool bwd = CARVE_STEP_IS_BWD(st);
      const int m = CARVE_STEP_TILE(st);
      // re-derive the lane coordinates inside the loop so per-lane addresses are
      // formed next to their use instead of being hoisted out of the loops
      int lane_ = threadIdx.x & 63;
      asm volatile("" : "+v"(lane_));
      const int g = lane_ >> 4, c = lane_ & 15, lane = lane_;
      const int t0 = ch * L + m * BLW;
      __syncthreads();  // previous users of the transient buffers are done
      // ---- B0: tile inputs from the prefetch registers --------------------------
      // the tile step processed after this one (this chunk or the previous one)
      int nch_ = ch, nst_ = st + 1;
      if (nst_ == nsteps) {
        nch_ = ch - 1;
        nst_ = 0;
      }
      const int nt0 = nch_ * L + CARVE_STEP_TILE(nst_) * BLW;
      {
        for (int u = 0; u < NQV; ++u) {
          const int x = tid + u * NT;
          if ((BLW * D / VEC) % NT != 0 && x >= BLW * D / VEC) break;
          const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;
          *reinterpret_cast<f32x4*>(sQ + t * LDD + j) = pq[u];
          *reinterpret_cast<f32x4*>(sK + t * LDD + j) = pk[u];
          if (bwd) {
            *reinterpret_cast<f32x4*>(sdO + t * LDD + j) = pdo[u];
            const T* rv = reinterpret_cast<const T*>(&pdo[u]);
            for (int e = 0; e < VEC; ++e) sdOT[(j + e) * LDB + t] = rv[e];
          }
        }
        if (tid < BLW) sBeta[tid] = pbeta;
        if (nch_ >= 0) CARVE_BWD_PREFETCH_VEC(nt0, CARVE_STEP_IS_BWD(nst_));
        for (int cq = 0; cq < CPW; ++cq)
          for (int it = 0; it < NIT; ++it) {
            store_tile(sS, LDD, 16 * it, 16 * (w * CPW + cq), S[cq][it], lane);
            if (bwd) store_tile(sdS, LDD, 16 * it, 16 * (w * CPW + cq), dS[cq][it], lane);
          }
      }
      __syncthreads();
      // ---- R1: tau = tanh(Q F^T) --------------------------------------------------
      for (int rt = w; rt < NRT; rt += NW) {
        f32x4 acc = zero4();
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          acc = M::mma(M::load(sQ + c * LDD + kofs), M::load(sF + (16 * rt + c) * LDD + kofs), acc);
        }
        for (int r = 0; r < 4; ++r) acc[r] = tanh_f(acc[r]);
        store_tile(sTau, LDR, 0, 16 * rt, acc, lane);
      }
      __syncthreads();
      // ---- R2: gates and retention factors ------------------------------------------
      float qv[CPW][4], kv[CPW][4], vv[CPW][4];
      float E[CPW][4], Ep[CPW][4], en[CPW][4], bgt[CPW][4], wgt[CPW][4], wv[CPW][4];
      float gam[CPW];
      float p[CPW][4];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        f32x4 accB = zero4(), accW = zero4();
        for (int ks = 0; ks < RP / KS; ++ks) {
          const int r0 = ks * KS + g * KPL;
          accB = M::mma(M::load(sTau + c * LDR + r0), fVb[cq][ks], accB);
          accW = M::mma(M::load(sTau + c * LDR + RP + r0), fVw[cq][ks], accW);
        }
        for (int r = 0; r < 4; ++r) {
          const float zb = cbx[cq][r] + accB[r];
          p[cq][r] = cg[cq][r] - softplus_f(zb);
          bgt[cq][r] = sigmoid_f(zb);
          wgt[cq][r] = sigmoid_f(cwx[cq][r] + accW[r]);
          vv[cq][r] = cv[cq][r];
          wv[cq][r] = wgt[cq][r] * vv[cq][r];
          qv[cq][r] = to_f(sQ[(4 * g + r) * LDD + jj]);
          kv[cq][r] = to_f(sK[(4 * g + r) * LDD + jj]);
        }
      }
      if (nch_ >= 0) CARVE_BWD_PREFETCH_GATES(nt0);
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        p[cq][1] += p[cq][0];
        p[cq][2] += p[cq][1];
        p[cq][3] += p[cq][2];
        float incl = p[cq][3];
        float y = __shfl_up(incl, 16);
        if (g >= 1) incl += y;
        y = __shfl_up(incl, 32);
        if (g >= 2) incl += y;
        const float excl = incl - p[cq][3];
        const float lam_end = __shfl(incl, 48 + c);
        for (int r = 0; r < 4; ++r) {
          const float lam = excl + p[cq][r];
          E[cq][r] = fast_exp(lam);
          en[cq][r] = fast_exp(-lam);
        }
        const float eprev = __shfl_up(E[cq][3], 16);
        Ep[cq][0] = g == 0 ? 1.0f : eprev;
        Ep[cq][1] = E[cq][0];
        Ep[cq][2] = E[cq][1];
        Ep[cq][3] = E[cq][2];
        gam[cq] = fast_exp(lam_end);
        f32x4 vK, vQ, vKi, vKh;
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * g + r;
          vK[r] = kv[cq][r] * Ep[cq][r];
          vQ[r] = qv[cq][r] * E[cq][r];
          vKi[r] = kv[cq][r] * en[cq][r];
          vKh[r] = vKi[r] * gam[cq];
          sK[t * LDD + jj] = (T)vK[r];
          sQ[t * LDD + jj] = (T)vQ[r];
          sKi[t * LDD + jj] = (T)vKi[r];
        }
        store_tile_t(sKT, LDB, 0, 16 * ct, vK, lane);
        store_tile_t(sQT, LDB, 0, 16 * ct, vQ, lane);
        store_tile_t(sKiT, LDB, 0, 16 * ct, vKi, lane);
        if (!bwd) store_tile_t(sKhT, LDB, 0, 16 * ct, vKh, lane);
        if (g == 0) sGam[jj] = gam[cq];
      }
      __syncthreads();
      // ---- R3: A, D, P and Ktil S^T ------------------------------------------------
      if (w == 0) {
        f32x4 accA = zero4(), accP = zero4();
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          const typename M::frag kb = M::load(sKi + c * LDD + kofs);
          accA = M::mma(M::load(sK + c * LDD + kofs), kb, accA);
          accP = M::mma(M::load(sQ + c * LDD + kofs), kb, accP);
        }
        f32x4 pv;
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * g + r;
          const float dval = (c < t) ? accA[r] : 0.0f;
          sDm[t * LDF + c] = dval;
          sA[t * LDF + c] = sBeta[t] * dval;
          pv[r] = (c <= t) ? accP[r] : 0.0f;
        }
        store_tile_t(sPT, LDB, 0, 0, pv, lane);
      }
      float Eerr[CPW][4];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        f32x4 acc = zero4();
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          acc = M::mma(M::load(sK + c * LDD + kofs), M::load(sS + (16 * ct + c) * LDD + kofs), acc);
        }
        f32x4 rv;
        for (int r = 0; r < 4; ++r) {
          Eerr[cq][r] = wv[cq][r] - acc[r];
          rv[r] = sBeta[4 * g + r] * Eerr[cq][r];
        }
        store_tile_t(sRT, LDB, 0, 16 * ct, rv, lane);
      }
      __syncthreads();
      // ---- R4: T = (I + A)^{-1}; du = Khat dS'^T + P^T dO ------------------------------
      if (w == 0 && g == 0) {
        float x[16];
        unit_lower_inverse_column(sA, LDF, c, x);
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          sTb[t * LDB + c] = (T)x[t];
          sTbT[c * LDB + t] = (T)x[t];
        }
      }
      if (bwd) {
        for (int cq = 0; cq < CPW; ++cq) {
          const int ct = w * CPW + cq;
          f32x4 acc = zero4();
          for (int ks = 0; ks < D / KS; ++ks) {
            const int kofs = ks * KS + g * KPL;
            acc = M::mma(M::load_scaled(sKi + c * LDD + kofs, sGam + kofs), M::load(sdS + (16 * ct + c) * LDD + kofs), acc);
          }
          acc = mma_k16<T>(acc, sPT + c * LDB, sdOT + (16 * ct + c) * LDB, g);
          store_tile_t(sduT, LDB, 0, 16 * ct, acc, lane);
        }
      }
      __syncthreads();
      // ---- R5: u = T R; dR = T^T du ---------------------------------------------------
      float dzw[CPW][4];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        const f32x4 u = mma_k16<T>(zero4(), sTb + c * LDB, sRT + (16 * ct + c) * LDB, g);
        if (bwd) {
          store_tile(sU, LDD, 0, 16 * ct, u, lane);
          const f32x4 dR = mma_k16<T>(zero4(), sTbT + c * LDB, sduT + (16 * ct + c) * LDB, g);
          f32x4 dE, dzv;
          for (int r = 0; r < 4; ++r) {
            const int t = 4 * g + r;
            dE[r] = sBeta[t] * dR[r];
            float db = dR[r] * Eerr[cq][r];
            db += __shfl_xor(db, 1);
            db += __shfl_xor(db, 2);
            db += __shfl_xor(db, 4);
            db += __shfl_xor(db, 8);
            if (c == 0) sDb[ct * BLW + t] = db;
            const float dwv = dE[r] * vv[cq][r];
            const int e = (t0 + t) * rs + jj;
            dv[e] = (T)(dE[r] * wgt[cq][r]);
            dzw[cq][r] = dwv * wgt[cq][r] * (1.0f - wgt[cq][r]);
            dwx[e] = (T)dzw[cq][r];
            dzv[r] = dzw[cq][r];
          }
          store_tile(sdR, LDD, 0, 16 * ct, dR, lane);
          store_tile(sdE, LDD, 0, 16 * ct, dE, lane);
          store_tile_t(sdET, LDB, 0, 16 * ct, dE, lane);
          store_tile(sdzw, LDD, 0, 16 * ct, dzv, lane);
        } else {
          store_tile_t(sUT, LDB, 0, 16 * ct, u, lane);
        }
      }
      __syncthreads();
      if (!bwd) {
        // forward tile: S <- S diag(gam) + u^T Khat, park it for the backward tiles
        f32x4* dst = reinterpret_cast<f32x4*>(a.substates + ((size_t)bh * msub + m + 1) * D * D) + (size_t)tid * CPW * NIT;
        for (int cq = 0; cq < CPW; ++cq) {
          const int ct = w * CPW + cq;
          for (int it = 0; it < NIT; ++it) {
            CARVE_SEQ();
            f32x4 acc;
            for (int r = 0; r < 4; ++r) acc[r] = S[cq][it][r] * gam[cq];
            acc = mma_k16<T>(acc, sUT + (16 * it + c) * LDB, sKhT + (16 * ct + c) * LDB, g);
            S[cq][it] = acc;
            if (m + 1 < msub - 1) dst[cq * NIT + it] = acc;  // the last one stays in registers
          }
        }
        continue;
      }
      // ---- G3: dKtil = -dE S, dQtil = dO S, dKhat = u dS'; dP, dA -------------------
      f32x4 dKt[CPW], dQt[CPW], dKh[CPW];
      float cs[CPW];
      for (int cq = 0; cq < CPW; ++cq) {
        dKt[cq] = mma_regB<T, NIT>(zero4(), sdE + c * LDD, S[cq], g);
        for (int r = 0; r < 4; ++r) dKt[cq][r] = -dKt[cq][r];
        dQt[cq] = mma_regB<T, NIT>(zero4(), sdO + c * LDD, S[cq], g);
        dKh[cq] = mma_regB<T, NIT>(zero4(), sU + c * LDD, dS[cq], g);
        float s_ = 0.0f;  // colsum(S * dS') for this column
        for (int it = 0; it < NIT; ++it)
          for (int r = 0; r < 4; ++r) s_ += S[cq][it][r] * dS[cq][it][r];
        s_ += __shfl_xor(s_, 16);
        s_ += __shfl_xor(s_, 32);
        cs[cq] = s_;
      }
      // S is dead for this tile: fetch the start state of the next backward tile
      {
        const float* src = nullptr;
        bool lane_major = false;
        if (m > 0) {
          if (m - 1 == 0) src = a.S_chunks + ((size_t)bh * nch + ch) * D * D;
          else {
            src = a.substates + ((size_t)bh * msub + m - 1) * D * D;
            lane_major = true;
          }
        } else if (ch > 0) {
          src = a.S_chunks + ((size_t)bh * nch + ch - 1) * D * D;
        }
        if (src) {
          if (lane_major) {
            const f32x4* sp = reinterpret_cast<const f32x4*>(src) + (size_t)tid * CPW * NIT;
            for (int cq = 0; cq < CPW; ++cq)
              for (int it = 0; it < NIT; ++it) S[cq][it] = sp[cq * NIT + it];
          } else {
            for (int cq = 0; cq < CPW; ++cq) {
              const int col = 16 * (w * CPW + cq) + c;
              for (int it = 0; it < NIT; ++it)
                for (int r = 0; r < 4; ++r) S[cq][it][r] = src[(size_t)(16 * it + 4 * g + r) * D + col];
            }
          }
        }
      }
      if (w == 0) {
        f32x4 acc = zero4();
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          acc = M::mma(M::load(sdO + c * LDD + kofs), M::load(sU + c * LDD + kofs), acc);
        }
        for (int r = 0; r < 4; ++r) acc[r] = (c <= 4 * g + r) ? acc[r] : 0.0f;
        store_tile(sdP, LDB, 0, 0, acc, lane);
        store_tile_t(sdPT, LDB, 0, 0, acc, lane);
      }
      if (w == (NW > 1 ? 1 : 0)) {
        f32x4 acc = zero4();
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          acc = M::mma(M::load(sdR + c * LDD + kofs), M::load(sU + c * LDD + kofs), acc);
        }
        f32x4 ddv;
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * g + r;
          const float dA = (c < t) ? -acc[r] : 0.0f;
          ddv[r] = sBeta[t] * dA;
          float db = dA * sDm[t * LDF + c];
          db += __shfl_xor(db, 1);
          db += __shfl_xor(db, 2);
          db += __shfl_xor(db, 4);
          db += __shfl_xor(db, 8);
          if (c == 0) sDb2[t] = db;
        }
        store_tile(sdD, LDB, 0, 0, ddv, lane);
        store_tile_t(sdDT, LDB, 0, 0, ddv, lane);
      }
      __syncthreads();
      // ---- G5: factored-pair gradients, dLam, gate-logit gradients -----------------
      float dqv[CPW][4], dkv[CPW][4], dzb[CPW][4];
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        const f32x4 dAq = mma_k16<T>(zero4(), sdD + c * LDB, sKiT + (16 * ct + c) * LDB, g);
        const f32x4 dPq = mma_k16<T>(zero4(), sdP + c * LDB, sKiT + (16 * ct + c) * LDB, g);
        f32x4 dcol = mma_k16<T>(zero4(), sdDT + c * LDB, sKT + (16 * ct + c) * LDB, g);
        dcol = mma_k16<T>(dcol, sdPT + c * LDB, sQT + (16 * ct + c) * LDB, g);
        float aL[4], pL[4], xs = 0.0f;
        for (int r = 0; r < 4; ++r) {
          const float gq = dQt[cq][r] * E[cq][r] + E[cq][r] * dPq[r];   // dq from Qtil and P
          const float gkh = dKh[cq][r] * gam[cq] * en[cq][r];           // dk from Khat
          const float gkc = en[cq][r] * dcol[r];                        // dk from the column side
          const float gkr = dKt[cq][r] * Ep[cq][r] + Ep[cq][r] * dAq[r];  // dk from Ktil and A's row side
          dqv[cq][r] = gq;
          dkv[cq][r] = gkr + gkh + gkc;
          aL[r] = qv[cq][r] * gq - kv[cq][r] * gkc - kv[cq][r] * gkh;
          pL[r] = kv[cq][r] * gkr;
          xs += kv[cq][r] * gkh;
        }
        xs += __shfl_xor(xs, 16);
        xs += __shfl_xor(xs, 32);
        if (g == 3) aL[3] += xs + cs[cq] * gam[cq];
        const float pnext = __shfl_down(pL[0], 16);
        float dLam[4];
        dLam[0] = aL[0] + pL[1];
        dLam[1] = aL[1] + pL[2];
        dLam[2] = aL[2] + pL[3];
        dLam[3] = aL[3] + (g < 3 ? pnext : 0.0f);
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
        const float after = tot - sfx[0];
        f32x4 dzv;
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * g + r;
          const float dl = sfx[r] + after;
          const int e = (t0 + t) * rs + jj;
          dgo[e] = dl;
          dzb[cq][r] = -dl * bgt[cq][r];
          dbx[e] = (T)dzb[cq][r];
          dzv[r] = dzb[cq][r];
        }
        store_tile(sdzb, LDD, 0, 16 * ct, dzv, lane);
        // dVb += dz_b^T tau_b, dVw += dz_w^T tau_w (A from registers, K = 16 tokens)
        for (int rt = 0; rt < NVT; ++rt) {
          if constexpr (sizeof(T) == 2) {
            typename M::frag ab, aw, bb, bw;
            for (int e = 0; e < 4; ++e) {
              ab[e] = (T)dzb[cq][e];
              aw[e] = (T)dzw[cq][e];
              bb[e] = sTau[(4 * g + e) * LDR + 16 * rt + c];
              bw[e] = sTau[(4 * g + e) * LDR + RP + 16 * rt + c];
              ab[4 + e] = (T)0.0f;
              aw[4 + e] = (T)0.0f;
              bb[4 + e] = (T)0.0f;
              bw[4 + e] = (T)0.0f;
            }
            dVb[cq][rt] = M::mma(ab, bb, dVb[cq][rt]);
            dVw[cq][rt] = M::mma(aw, bw, dVw[cq][rt]);
          } else {
            for (int r = 0; r < 4; ++r) {
              dVb[cq][rt] = M::mma(dzb[cq][r], sTau[(4 * g + r) * LDR + 16 * rt + c], dVb[cq][rt]);
              dVw[cq][rt] = M::mma(dzw[cq][r], sTau[(4 * g + r) * LDR + RP + 16 * rt + c], dVw[cq][rt]);
            }
          }
        }
      }
      __syncthreads();
      // ---- G8: dtau = dz V, dY = dtau (1 - tau^2) ------------------------------------
      for (int gi = 0; gi < NGT; ++gi) {
        const int x = w + gi * NW;
        if (x >= 2 * NVT) break;
        const int half = x / NVT, rt = x % NVT;
        const T* arow = (half ? sdzw : sdzb) + c * LDD;
        f32x4 acc = zero4();
        for (int ks = 0; ks < D / KS; ++ks) acc = M::mma(M::load(arow + ks * KS + g * KPL), fVt[gi][ks], acc);
        f32x4 dy;
        for (int r = 0; r < 4; ++r) {
          const float tv = to_f(sTau[(4 * g + r) * LDR + half * RP + 16 * rt + c]);
          dy[r] = acc[r] * (1.0f - tv * tv);
        }
        store_tile(sdY, LDR, 0, half * RP + 16 * rt, dy, lane);
        store_tile_t(sdYT, LDB, 0, half * RP + 16 * rt, dy, lane);
      }
      __syncthreads();
      // ---- G9: dq += dY F, outputs, dF += dY^T q, dS <- ... -----------------------------
      for (int cq = 0; cq < CPW; ++cq) {
        const int ct = w * CPW + cq;
        const int jj = 16 * ct + c;
        f32x4 acc = zero4();
        for (int ks = 0; ks < R2 / KS; ++ks) {
          const int r0 = ks * KS + g * KPL;
          typename M::frag bfg;
          if constexpr (KPL == 8) {
            for (int e = 0; e < 8; ++e) bfg[e] = sF[(r0 + e) * LDD + jj];
          } else {
            bfg = sF[r0 * LDD + jj];
          }
          acc = M::mma(M::load(sdY + c * LDR + r0), bfg, acc);
        }
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * g + r;
          const int e = (t0 + t) * rs + jj;
          dq[e] = (T)(dqv[cq][r] + acc[r]);
          dk[e] = (T)dkv[cq][r];
        }
        for (int rt = 0; rt < NRT; ++rt) {
          if constexpr (sizeof(T) == 2) {
            typename M::frag af, bfg;
            for (int e = 0; e < 4; ++e) {
              af[e] = sdYT[(16 * rt + c) * LDB + 4 * g + e];
              bfg[e] = (T)qv[cq][e];
              af[4 + e] = (T)0.0f;
              bfg[4 + e] = (T)0.0f;
            }
            dF[cq][rt] = M::mma(af, bfg, dF[cq][rt]);
          } else {
            for (int r = 0; r < 4; ++r)
              dF[cq][rt] = M::mma(sdYT[(16 * rt + c) * LDB + 4 * g + r], qv[cq][r], dF[cq][rt]);
          }
        }
        for (int it = 0; it < NIT; ++it) {
          CARVE_SEQ();
          f32x4 acc1, acc2;
          for (int r = 0; r < 4; ++r) acc1[r] = dS[cq][it][r] * gam[cq];
          acc1 = mma_k16<T>(acc1, sdOT + (16 * it + c) * LDB, sQT + (16 * ct + c) * LDB, g);
          acc2 = mma_k16<T>(zero4(), sdET + (16 * it + c) * LDB, sKT + (16 * ct + c) * LDB, g);
          for (int r = 0; r < 4; ++r) dS[cq][it][r] = acc1[r] - acc2[r];
        }
      }
      if (w == 0 && lane < BLW) {
        float db = sDb2[lane];
        for (int x = 0; x < NCT; ++x) db += sDb[x * BLW + lane];
        dbeta[(t0 + lane) * H] = (T)db;
      }
    }  // tile steps

    // ---- chunk start: glue through the folded read-out ------------------------------
    __syncthreads();
    for (int cq = 0; cq < CPW; ++cq)
      for (int rt = 0; rt < NRT; ++rt) store_tile(sdF, LDD, 16 * rt, 16 * (w * CPW + cq), dF[cq][rt], lane);
    // dS += [Ub;Uw]^T dF  (contraction over the rows of dF, held in registers)
    for (int cq = 0; cq < CPW; ++cq)
      for (int it = 0; it < NIT; ++it) {
        CARVE_SEQ();
        f32x4 acc = dS[cq][it];
        const T* urow = UT + (size_t)(16 * it + c) * R2;  // value row this lane supplies as A
        if constexpr (KPL == 8) {
          for (int ks = 0; ks < R2 / 32; ++ks) {
            typename M::frag af, bfg;
            const bf16x4 lo = *reinterpret_cast<const bf16x4*>(urow + 32 * ks + 4 * g);
            const bf16x4 hi = *reinterpret_cast<const bf16x4*>(urow + 32 * ks + 16 + 4 * g);
            for (int e = 0; e < 4; ++e) {
              af[e] = lo[e];
              af[4 + e] = hi[e];
              bfg[e] = (T)dF[cq][2 * ks][e];
              bfg[4 + e] = (T)dF[cq][2 * ks + 1][e];
            }
            acc = M::mma(af, bfg, acc);
          }
        } else {
          for (int rt = 0; rt < NRT; ++rt)
            for (int r4 = 0; r4 < 4; ++r4) acc = M::mma(urow[16 * rt + 4 * g + r4], dF[cq][rt][r4], acc);
        }
        dS[cq][it] = acc;
      }
    __syncthreads();
    // d[Ub;Uw] += dF S_hat^T  (sS still holds S_hat from the chunk's first tile)
    for (int cq = 0; cq < CPW; ++cq) {
      const int ct = w * CPW + cq;
      for (int rt = 0; rt < NRT; ++rt) {
        CARVE_SEQ();
        f32x4 acc = dU[cq][rt];
        for (int ks = 0; ks < D / KS; ++ks) {
          const int kofs = ks * KS + g * KPL;
          acc = M::mma(M::load(sdF + (16 * rt + c) * LDD + kofs), M::load(sS + (16 * ct + c) * LDD + kofs), acc);
        }
        dU[cq][rt] = acc;
      }
    }
  }  // chunks

  if (a.dS0) {
    for (int cq = 0; cq < CPW; ++cq) {
      const int col = 16 * (w * CPW + cq) + c;
      for (int it = 0; it < NIT; ++it)
        for (int r = 0; r < 4; ++r) a.dS0[soff + (size_t)(16 * it + 4 * g + r) * D + col] = dS[cq][it][r];
    }
  }
  float* part = a.part + (size_t)bh * part_floats(R, D);
  float* pUb = part;
  float* pUw = part + (size_t)R * D;
  float* pVb = part + (size_t)2 * R * D;
  float* pVw = part + (size_t)3 * R * D;
  for (int cq = 0; cq < CPW; ++cq) {
    const int ct = w * CPW + cq;
    for (int rt = 0; rt < NRT; ++rt)
      for (int r = 0; r < 4; ++r) {
        const int rr = 16 * rt + 4 * g + r;
        if (rr < R) pUb[(size_t)rr * D + 16 * ct + c] = dU[cq][rt][r];
        else if (rr >= RP && rr < RP + R) pUw[(size_t)(rr - RP) * D + 16 * ct + c] = dU[cq][rt][r];
      }
    for (int rt = 0; rt < NVT; ++rt)
      for (int r = 0; r < 4; ++r) {
        const int j = 16 * ct + 4 * g + r, col = 16 * rt + c;
        if (col < R) {
          pVb[(size_t)j * R + col] = dVb[cq][rt][r];
          pVw[(size_t)j * R + col] = dVw[cq][rt][r];
        }
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
template <typename T, int D, int RP>
static int launch_bwd_t(const BwdArgs& a, hipStream_t stream) {
  const BwdLds lay = bwd_lds<T, D>(RP);
  auto kern = carve_bwd_kernel<T, D, RP>;
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lay.total) != hipSuccess)
      return CARVE_ERR_HIP;
    attr_set = true;
  }
  const int n = 2 * RP * D;
  hipLaunchKernelGGL(carve_pack_u_kernel<T>, dim3((n + 255) / 256), dim3(256), 0, stream, a.Ub, a.Uw, a.R, RP, D,
                     reinterpret_cast<T*>(const_cast<void*>(a.Up)), reinterpret_cast<T*>(const_cast<void*>(a.UT)));
  if (hipGetLastError() != hipSuccess) return CARVE_ERR_HIP;
  hipLaunchKernelGGL(kern, dim3(a.B * a.H), dim3(bwd_threads(D)), lay.total, stream, a);
  return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
}

template <typename T, int D>
static int launch_bwd_r(const BwdArgs& a, hipStream_t s) {
  if (a.RP == 32) return launch_bwd_t<T, D, 32>(a, s);
  if (a.RP == 64) return launch_bwd_t<T, D, 64>(a, s);
  return CARVE_ERR_UNSUPPORTED;
}

int launch_bwd(const BwdArgs& a, int dtype, int D, int LW, hipStream_t s) {
  if (LW != BLW) return CARVE_ERR_UNSUPPORTED;
  if (dtype == CARVE_BF16) {
    if (D == 32) return launch_bwd_r<bf16_t, 32>(a, s);
    if (D == 64) return launch_bwd_r<bf16_t, 64>(a, s);
    if (D == 128 && a.RP == 32) return launch_bwd_t<bf16_t, 128, 32>(a, s);
  } else {
    if (D == 32) return launch_bwd_r<float, 32>(a, s);
    if (D == 64 && a.RP == 32) return launch_bwd_t<float, 64, 32>(a, s);
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
