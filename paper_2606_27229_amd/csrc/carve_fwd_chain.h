// carve_fwd_chain.h -- chunked CARVE forward on gfx950: one workgroup per
// (batch, head) runs the whole sequence as a persistent chain of WY blocks.
// (Kernel templates; every variant is instantiated in a translation unit of its
// own, carve_variant.hip.)
//
// A gate chunk (L tokens) is evaluated as L / WB WY blocks of WB <= 64 tokens
// (WB = L for L <= 64).  At the start of every chunk the state S_hat is folded
// once (Eq. content_readout); every block of the chunk uses the same fold:
//   F = [Ub; Uw] S_hat,  tau = tanh(q F^T),
//   z_b = bx + tau_b Vb^T,  z_w = wx + tau_w Vw^T            (Eq. erase_gate)
//   l = g - softplus(z_b) = log(exp(g) (1 - sigmoid(z_b))),   w = sigmoid(z_w)
// Inside a block, with lam the prefix sums of l from the block start (lam_{-1}
// = 0), c_i = lam at the end of 16-token tile i (c_{-1} = 0), S the block start
// state and the WY form of Sec. WY-form intra-chunk solve re-derived from the
// recurrence of Eq. carve_state, the exponentials of a token in tile i are
// taken relative to a per-key-channel reference m_i:
//   Kt_t = k_t e^{lam_{t-1} - m_i},  Qt_t = q_t e^{lam_t - m_i},  Ki_t = k_t e^{m_i - lam_t}
//   A_ts = beta_t Kt_t . Ki_s e^{m_i - m_j},  P_ts = Qt_t . Ki_s e^{m_i - m_j}   (s in tile j)
//   u = (I + A)^{-1} beta (w * v - Kt diag(e^{m_i}) S^T)          (corrected values)
//   o = Qt diag(e^{m_i}) S^T + P u
//   S <- S diag(e^{lam_end}) + sum_s u_s (Ki_s e^{lam_end - m_j})^T
// (= S diag(e^{lam_end}) + sum_s u_s k_s^T e^{lam_end - lam_s}).
// A key channel that keeps lam_end >= -kWideLog over the block takes one
// reference for every tile, m_i = lam_end / 2 (the middle of the block's
// log-retention range; no factor exceeds e^{kWideLog / 2}); any other channel
// takes the middle of each tile's own range, m_i = (c_{i-1} + c_i) / 2.  While
// every channel of the block has one reference (a flag per wave, combined
// across the workgroup after a barrier) the pair factors are 1, the state
// factors the one e^{lam_end / 2}, and the products run on the stored
// operands.  Otherwise every product across tiles is formed from operands that
// do not exceed the raw token values: for i > j, Ki_s e^{c_j - m_j} against
// Kt_t (Qt_t) e^{m_i - c_j} (the latter e^{c_i - m_i} for adjacent tiles), and
// the state update scales Ki_s by e^{lam_end - m_j}; these factors are 1 on
// one-reference channels.  The factors are per-channel tables in LDS
// (fwd_tab_rows).
// The unit-lower-triangular solve is blocked over 16-token tiles: the diagonal
// tiles are inverted by substitution, the off-diagonal coupling is applied on
// the matrix cores while walking the tiles in order.
//
// Wave w owns the 16-wide tile w of the value axis (state rows, values, u, o)
// and the 16-wide tile w of the key axis (gate arithmetic, decayed keys).  The
// state lives in registers in the matrix-core result layout for the whole call.
//
// Memory: the next block's token data is loaded into registers while the
// current block runs (q, k and bx as whole rows, 16 bytes per lane, then
// staged through LDS; a wave load that touches 16 token rows for 32 bytes
// each streams at well under half the rate); each block starts with one wait
// for all of this wave's outstanding memory operations, by then at least half
// a block old.  The
// output of a block is stored at the start of the next block, so no wait on
// the chain ever covers a store that was just issued.
//
// With the scalar write gate (kVarScalarW) the fold has the Ub rows only, the
// write logit of a token is one scalar per head, staged with beta, and w v is
// that gate times v.  With the input activations (kVarAct) q, k and v arrive
// raw: the rows of q and k are staged as SiLU(raw) / |SiLU(raw)| (the norm
// summed over the row's lanes while staging), v as SiLU(raw).
//
// Precondition (not checked): the log retention summed over every 16-token
// tile stays above about -150 per key channel (blocks of a single tile: -170).
// Tile factors up to e^{|tile sum| / 2} are formed in f32 and the token dtype;
// where e^{m_i} S falls below the normal range, what is lost is below
// e^{|tile sum| / 2 - 87} of the state's contribution.
#pragma once
#include "carve_kernels.h"

namespace carve {

// Tile x of a row-major enumeration of the lower-triangular tiles (i, j):
// strict (j < i, starting at i = 1) or inclusive (j <= i).
__host__ __device__ constexpr int tri_row(int x, bool strict) {
  int i = strict ? 1 : 0;
  while (x >= (strict ? i : i + 1)) {
    x -= strict ? i : i + 1;
    ++i;
  }
  return i;
}
__host__ __device__ constexpr int tri_col(int x, bool strict) {
  int i = strict ? 1 : 0;
  while (x >= (strict ? i : i + 1)) {
    x -= strict ? i : i + 1;
    ++i;
  }
  return x;
}
static_assert(tri_row(0, true) == 1 && tri_col(0, true) == 0 && tri_row(5, true) == 3 && tri_col(5, true) == 2, "");
static_assert(tri_row(0, false) == 0 && tri_row(2, false) == 1 && tri_col(2, false) == 1 && tri_col(9, false) == 3, "");

// q * f (per-element factors at p), rounded back to the operand type
template <typename T>
__device__ __forceinline__ typename Quad<T>::q scale_q(typename Quad<T>::q q, const float* p) {
  return Quad<T>::cvt(Quad<T>::f32(q) * *reinterpret_cast<const f32x4*>(p));
}

// GATED: the decay g is formed in the kernel from its raw logit f (token
// dtype) as -exp(A) softplus(f + tau_f) (Eq. decay_gate, Sec. decay_gate),
// with A and tau_f of the head held in LDS.
template <typename T, int D, int WB, int RP, int VAR>
__global__ void __launch_bounds__(fwd_threads(D)) carve_chain_fwd_kernel(FwdArgs a) {
  typedef Quad<T> Qd;
  typedef typename Qd::q quad;
  constexpr bool GATED = (VAR & kVarGated) != 0;
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr bool ACT = (VAR & kVarAct) != 0;
  constexpr int NT = fwd_threads(D);
  constexpr int NW = NT / 64;
  constexpr int NJT = D / 16;
  constexpr int NB = WB / 16;
  constexpr int R2 = fold_rows(RP, VAR);   // rows of the fold
  constexpr int NRT = R2 / 16;
  constexpr int NRB = RP / 16;
  // bf16 operand tiles: rows of 16 (mod 32) elements with quad q of row r at
  // q ^ ((r >> 2) & 3) (qswz; CARVE_QX below), bank-conflict-free for their
  // row-wise, paired row-wise and transposing reads and their quad writes;
  // f32 tiles: 16-byte row pad, no swizzle
  constexpr int LDD = fwd_qstride<T>(D), LDR = fwd_qstride<T>(R2), LDW = fwd_qstride<T>(WB),
                LDB = fwd_qstride<T>(16);
  constexpr int NTA = NB * (NB - 1) / 2;   // off-diagonal tiles of A
  constexpr int NTP = NB * (NB + 1) / 2;   // tiles of P
  // coupling step: NDW waves (one per SIMD) take the diagonal inverses, NOW
  // waves the off-diagonal tiles (all waves when each has a diagonal tile)
  constexpr int NDW = NB < NW ? NB : NW;
  constexpr int NOW = NW > NDW ? NW - NDW : NW;
  constexpr bool kSplitRoles = NOW < NW;
  static_assert(NW == NJT && NW >= 2, "one wave per 16-wide tile, at least two waves");
  static_assert(D % 32 == 0, "K32 steps over the key / value axis");

  const int tid = threadIdx.x, lane = tid & 63;
#define CARVE_QX(R_) qswz<T>(R_)
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  const int g = lane >> 4, c = lane & 15;
  const int H = a.H, Tn = a.T, L = a.L, R = a.R;
  const int nblk = Tn / WB, bpc = L / WB;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr ChainLds lay = chain_lds<T, D, WB, RP, VAR>();
  T* sU = reinterpret_cast<T*>(smem + lay.U);      // [R2][LDD]   [Ub; 0; Uw; 0] or [Ub; 0]
  T* sS = reinterpret_cast<T*>(smem + lay.X);      // [D][LDD]    S_hat[v][j]
  T* sKt = reinterpret_cast<T*>(smem + lay.Kt);    // [WB][LDD]   (aliases sS)
  T* sBx = reinterpret_cast<T*>(smem + lay.Bx);    // [WB][LDD]   raw bx (aliases sS)
  T* sKi = reinterpret_cast<T*>(smem + lay.Ki);    // [WB][LDD]   raw k, then Ki
  T* sF = reinterpret_cast<T*>(smem + lay.F);      // [R2][LDD]   F[r][j]
  T* sQ = reinterpret_cast<T*>(smem + lay.Q);      // [WB][LDD]   raw q, then Qt
  T* sTau = reinterpret_cast<T*>(smem + lay.Tau);  // [WB][LDR]   tau[t][r]
  T* sA = reinterpret_cast<T*>(smem + lay.A);      // [WB][LDW]   -A[t][s] (off-diagonal tiles)
  T* sP = reinterpret_cast<T*>(smem + lay.P);      // [WB][LDW]   P[t][s]
  T* sTmT = reinterpret_cast<T*>(smem + lay.TmT);          // [NB][16][LDB] T_ii[t][s] at (s, t)
  // factor tables [fwd_tab_rows(NB)][D]: rows kTabSt + i = e^{m_i}, kTabUp + i =
  // e^{lam_end - m_i}, kTabHalf + i = e^{c_i - m_i}, kTabEnd = e^{lam_end},
  // kTabGap + (i - 2)(i - 1) / 2 + j = e^{m_i - c_j} (i >= j + 2); a block with
  // one reference per channel writes only row kTabSt
  float* sTab = reinterpret_cast<float*>(smem + lay.Tab);
  constexpr int kTabSt = 0, kTabUp = NB, kTabHalf = 2 * NB, kTabEnd = 3 * NB, kTabGap = 3 * NB + 1;
  constexpr int NTAB = fwd_tab_rows(NB);
  static_assert(NTAB <= 16, "one table row per lane of a 16-lane row");
  int* sFlag = reinterpret_cast<int*>(smem + lay.Flag);   // [NW]
  float* sBeta = reinterpret_cast<float*>(smem + lay.Beta);  // [2][WB] (block parity)
  float* sWs = sBeta + 2 * WB;                     // [2][WB] sigmoid(wx) (SW; block parity)
  constexpr bool SVW = chain_stage_vw<T, D, WB, RP, VAR>();
  T* sVW = reinterpret_cast<T*>(smem + lay.VW);    // [2][WB][D]  v, wx (swizzled; SVW; v only with SW)
  float* sGate = reinterpret_cast<float*>(smem + lay.Gate);  // [2][D] -exp(A), tau_f (GATED)

  const size_t bh0 = ((size_t)b * Tn * H + h) * D;
  const size_t bh1 = (size_t)b * Tn * H + h;
  const int rs = H * D;
  const T* __restrict__ q = reinterpret_cast<const T*>(a.q) + bh0;
  const T* __restrict__ k = reinterpret_cast<const T*>(a.k) + bh0;
  const T* __restrict__ v = reinterpret_cast<const T*>(a.v) + bh0;
  const T* __restrict__ bx = reinterpret_cast<const T*>(a.bx) + bh0;
  const T* __restrict__ wx = reinterpret_cast<const T*>(a.wx) + (SW ? bh1 : bh0);
  const T* __restrict__ beta = reinterpret_cast<const T*>(a.beta) + bh1;
  const float* __restrict__ gl = GATED ? nullptr : a.g + bh0;
  const T* __restrict__ fl = GATED ? reinterpret_cast<const T*>(a.f) + bh0 : nullptr;
  T* __restrict__ o = reinterpret_cast<T*>(a.o) + bh0;

  // ---- shared parameters ------------------------------------------------------
  if (GATED)
    for (int x = tid; x < D; x += NT) {
      sGate[x] = -expf(a.A[h * D + x]);
      sGate[D + x] = a.tau_f[h * D + x];
    }
  for (int x = tid; x < R2 * D; x += NT) {
    const int rr = x / D, i = x % D;
    float u = 0.0f;
    if (rr < R) u = a.Ub[rr * D + i];
    else if (!SW && rr >= RP && rr < RP + R) u = a.Uw[(rr - RP) * D + i];
    sU[rr * LDD + (i ^ CARVE_QX(rr))] = (T)u;
  }
  // Vb / Vw operand quads, lane (g, c): V[16 w + c][16 ks + 4 g + e]
  quad fVb[NRB], fVw[NRB];
  for (int ks = 0; ks < NRB; ++ks) {
    f32x4 tb, tw;
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * ks + 4 * g + e;
      tb[e] = r < R ? a.Vb[(16 * w + c) * R + r] : 0.0f;
      tw[e] = (!SW && r < R) ? a.Vw[(16 * w + c) * R + r] : 0.0f;
    }
    fVb[ks] = Qd::cvt(tb);
    fVw[ks] = Qd::cvt(tw);
  }
  // identity operand, lane (g, c): I[4 g + e][c]
  quad fI;
  {
    f32x4 t;
    for (int e = 0; e < 4; ++e) t[e] = (4 * g + e == c) ? 1.0f : 0.0f;
    fI = Qd::cvt(t);
  }

  // ---- state: St[jt][e] = S[v = 16 w + c][j = 16 jt + 4 g + e] ----------------
  f32x4 St[NJT];
  const size_t soff = (size_t)bh * D * D;
  for (int jt = 0; jt < NJT; ++jt)
    St[jt] = a.S0 ? gload4(a.S0 + soff + (16 * w + c) * D + 16 * jt + 4 * g) : zero4();

  // ---- prefetch registers ---------------------------------------------------------
  // q, k, bx: whole rows, 16 bytes per lane (coalesced), staged through LDS;
  // g, v, wx: token tile bb as lane (g, c) = token 16 bb + c, elements 16 w + 4 g ..
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr int VEC = 16 / sizeof(T);                // elements per 16-byte vector
  constexpr int NVX = WB * D / VEC;                  // vectors of one [WB][D] tile
  constexpr int NXV = (NVX + NT - 1) / NT;           // per thread
  static_assert(NVX % 64 == 0, "whole waves of row chunks (the row sums run over lanes)");
  u32x4 cq[NXV], ck[NXV], cbx[NXV];
  quad pv[NB], pwx[NB];      // per-tile value-side operands (without SVW)
  u32x4 cv[NXV], cwx[NXV];   // whole rows of v and wx (with SVW)
  f32x4 pg[NB];     // g per tile (ungated)
  quad pf[NB];      // f per tile (GATED)
  T pbeta = (T)0.0f, pws = (T)0.0f;   // beta and (SW) the write logit of token lane % WB
#define CARVE_PREFETCH_Q(BLK_)                                                     \
  do {                                                                             \
    const int t0_ = (BLK_) * WB;                                                   \
    for (int u_ = 0; u_ < NXV; ++u_) {                                             \
      const int x_ = tid + u_ * NT;                                                \
      if (NVX % NT != 0 && x_ >= NVX) break;                                       \
      cq[u_] = *reinterpret_cast<const u32x4*>(q + (t0_ + x_ / (D / VEC)) * rs + (x_ % (D / VEC)) * VEC); \
    }                                                                              \
    if (w == 0) {                                                                  \
      pbeta = beta[(t0_ + (lane % WB)) * H];                                       \
      if constexpr (SW) pws = wx[(t0_ + (lane % WB)) * H];                         \
    }                                                                              \
  } while (0)
#define CARVE_PREFETCH_GATES(BLK_)                                                 \
  do {                                                                             \
    const int t0_ = (BLK_) * WB;                                                   \
    for (int u_ = 0; u_ < NXV; ++u_) {                                             \
      const int x_ = tid + u_ * NT;                                                \
      if (NVX % NT != 0 && x_ >= NVX) break;                                       \
      const int o_ = (t0_ + x_ / (D / VEC)) * rs + (x_ % (D / VEC)) * VEC;         \
      ck[u_] = *reinterpret_cast<const u32x4*>(k + o_);                            \
      cbx[u_] = *reinterpret_cast<const u32x4*>(bx + o_);                          \
    }                                                                              \
  } while (0)
  // per-tile operands of the gates (16 token rows of this wave's 16 columns)
#define CARVE_PREFETCH_G(BLK_)                                                     \
  do {                                                                             \
    int cs_ = c, gs_ = g;                                                          \
    asm volatile("" : "+v"(cs_), "+v"(gs_));                                       \
    for (int bb_ = 0; bb_ < NB; ++bb_) {                                           \
      const int e_ = ((BLK_) * WB + 16 * bb_ + cs_) * rs + 16 * w + 4 * gs_;      \
      if constexpr (GATED) pf[bb_] = Qd::ld(fl + e_);                              \
      else pg[bb_] = *reinterpret_cast<const f32x4*>(gl + e_);                     \
    }                                                                              \
  } while (0)
#define CARVE_PREFETCH_VW(BLK_)                                                    \
  do {                                                                             \
    if constexpr (SVW) {                                                           \
      const int t0_ = (BLK_) * WB;                                                 \
      for (int u_ = 0; u_ < NXV; ++u_) {                                           \
        const int x_ = tid + u_ * NT;                                              \
        if (NVX % NT != 0 && x_ >= NVX) break;                                     \
        const int o_ = (t0_ + x_ / (D / VEC)) * rs + (x_ % (D / VEC)) * VEC;       \
        cv[u_] = *reinterpret_cast<const u32x4*>(v + o_);                          \
        if constexpr (!SW) cwx[u_] = *reinterpret_cast<const u32x4*>(wx + o_);     \
      }                                                                            \
    } else {                                                                       \
      int cs_ = c, gs_ = g;                                                        \
      asm volatile("" : "+v"(cs_), "+v"(gs_));                                     \
      for (int bb_ = 0; bb_ < NB; ++bb_) {                                         \
        const int e_ = ((BLK_) * WB + 16 * bb_ + cs_) * rs + 16 * w + 4 * gs_;    \
        pv[bb_] = Qd::ld(v + e_);                                                  \
        if constexpr (!SW) pwx[bb_] = Qd::ld(wx + e_);                             \
      }                                                                            \
    }                                                                              \
  } while (0)
  // v / wx rows into VW: 16-byte chunk kk of row t goes to chunk kk ^ (t mod NC)
  // (a swizzle instead of padding: the 16 rows a wave reads with one quad load
  // fall into distinct banks)
  constexpr int NC = D / VEC;                        // 16-byte chunks per row
#define CARVE_STAGE_VW()                                                           \
  do {                                                                             \
    for (int u_ = 0; u_ < NXV; ++u_) {                                             \
      const int x_ = tid + u_ * NT;                                                \
      if (NVX % NT != 0 && x_ >= NVX) break;                                       \
      const int t_ = x_ / NC, kk_ = x_ % NC;                                       \
      T* d_ = sVW + t_ * D + (kk_ ^ (t_ & (NC - 1))) * VEC;                        \
      *reinterpret_cast<u32x4*>(d_) = ACT ? act_chunk<T>(cv[u_], 1.0f) : cv[u_];   \
      if constexpr (!SW) *reinterpret_cast<u32x4*>(d_ + WB * D) = cwx[u_];         \
    }                                                                              \
  } while (0)
  // (L2_: the rows are raw q or k, staged activated; a row's D / VEC chunks
  // sit in consecutive lanes of one wave, so its norm is a sum over them)
#define CARVE_STAGE_ROWS(DST_, SRC_, L2_)                                          \
  do {                                                                             \
    for (int u_ = 0; u_ < NXV; ++u_) {                                             \
      const int x_ = tid + u_ * NT;                                                \
      if (NVX % NT != 0 && x_ >= NVX) break;                                       \
      u32x4 r_ = (SRC_)[u_];                                                       \
      if constexpr (L2_) r_ = act_chunk<T>(r_, act_row_inv_norm<T, D / VEC>(r_));  \
      const int row_ = x_ / (D / VEC), q2_ = (x_ % (D / VEC)) * 2;                 \
      /* the chunk's quads 2m, 2m + 1 go to quads (2m, 2m + 1) ^ h: the pair    \
         moves by h & 2 and its halves swap when h & 1 (bf16, VEC = 8) */       \
      const int h_ = CARVE_QX(row_) >> 2;                                          \
      if (sizeof(T) == 2 && (h_ & 1)) r_ = u32x4{r_[2], r_[3], r_[0], r_[1]};      \
      *reinterpret_cast<u32x4*>((DST_) + row_ * LDD + (sizeof(T) == 2 ? ((q2_ ^ (h_ & 2)) * 4) : q2_ * 2)) = r_; \
    }                                                                              \
  } while (0)
  CARVE_PREFETCH_Q(0);
  CARVE_PREFETCH_GATES(0);
  CARVE_PREFETCH_G(0);
  CARVE_PREFETCH_VW(0);

  quad oq[NB];   // o of the previous block, lane (g, c): o[t = 16 bb + c][v = 16 w + 4 g + e]
  int oprev = -1;

  for (int blk = 0; blk < nblk; ++blk) {
    const int t0 = blk * WB;
    const bool cstart = (blk % bpc) == 0;
    const int par = blk & 1;

    // ---- stage: wait for the prefetch; chunk start state --------------------------
    // The block's global stores and the next block's loads are spread over the
    // steps that use only LDS and the matrix cores (fold, tau, coupling,
    // substitution): issued in one burst they would stall every wave behind
    // the CU's memory pipeline.  Store addresses come from opaque lane
    // coordinates, recomputed where needed instead of held across the loop.
  // The chunk start state goes out in whole 128-byte lines: for the column
  // tiles 2m and 2m + 1, neighbouring lanes c and c ^ 1 (rows 2r and 2r + 1)
  // swap one quad each, so that one store writes row 2r (tile 2m from the even
  // lane, tile 2m + 1 from the odd one) and the next row 2r + 1.  Tiles
  // [JT0_ / 2 * 2, JT1_ / 2 * 2) are stored.
#define CARVE_STORE_S(JT0_, JT1_)                                                  \
    do {                                                                           \
      if (cstart && a.S_chunks) {                                                  \
        int cs_ = c, gs_ = g;                                                      \
        asm volatile("" : "+v"(cs_), "+v"(gs_));                                   \
        const bool odd_ = (cs_ & 1) != 0;                                          \
        float* r0_ = a.S_chunks + ((size_t)bh * (Tn / L) + blk / bpc) * D * D + (16 * w + (cs_ & ~1)) * D + 4 * gs_ + (odd_ ? 16 : 0); \
        for (int m_ = (JT0_) / 2; m_ < (JT1_) / 2; ++m_) {                         \
          f32x4 st0_, st1_;                                                        \
          for (int e_ = 0; e_ < 4; ++e_) {                                         \
            const float rv_ = lane_xor1(odd_ ? St[2 * m_][e_] : St[2 * m_ + 1][e_]); \
            st0_[e_] = odd_ ? rv_ : St[2 * m_][e_];                                \
            st1_[e_] = odd_ ? St[2 * m_ + 1][e_] : rv_;                            \
          }                                                                        \
          *reinterpret_cast<f32x4*>(r0_ + 32 * m_) = st0_;                         \
          *reinterpret_cast<f32x4*>(r0_ + D + 32 * m_) = st1_;                     \
        }                                                                          \
      }                                                                            \
    } while (0)
    vm_wait_all();
    if (cstart) {
      for (int jt = 0; jt < NJT; ++jt) Qd::st(sS + (16 * w + c) * LDD + 16 * jt + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(St[jt]));
    }
    CARVE_STAGE_ROWS(sQ, cq, ACT);
    if (w == 0 && lane < WB) {
      sBeta[par * WB + lane] = (float)pbeta;
      if constexpr (SW) sWs[par * WB + lane] = sigmoid_f((float)pws);
    }
    {
      const int nx = blk + 1 < nblk ? blk + 1 : blk;
      CARVE_PREFETCH_Q(nx);
    }
    __syncthreads();
    // the chunk start state goes out in two halves, the second during the
    // coupling step; the off-diagonal workers, whose chains bound that step,
    // store all of theirs here
    CARVE_STORE_S(0, kSplitRoles && w < NOW ? NJT : NJT / 2);
    // raw keys of the block into free LDS (read by the gates)
    CARVE_STAGE_ROWS(sKi, ck, ACT);
    if constexpr (SVW) CARVE_STAGE_VW();

    // ---- fold F^T[j][r] = sum_v S_hat[v][j] U[r][v] (key tile w) --------------
    if (cstart) {
      // the state's column block (this wave's key tile) is read once per
      // 32-value step and serves every fold row tile
      f32x4 acc[NRT];
      for (int rt = 0; rt < NRT; ++rt) acc[rt] = zero4();
      for (int vp = 0; vp < D / 32; ++vp) {
        const quad a0 = Qd::ld_tr_sw(sS, LDD, 32 * vp, 16 * w, g, c);
        const quad a1 = Qd::ld_tr_sw(sS, LDD, 32 * vp + 16, 16 * w, g, c);
        for (int rt = 0; rt < NRT; ++rt) {
          const T* ur = sU + (16 * rt + c) * LDD + 32 * vp + ((4 * g) ^ CARVE_QX(c));
          acc[rt] = Qd::mma32(a0, a1, Qd::ld(ur), Qd::ld(ur + 16), acc[rt]);
        }
      }
      for (int rt = 0; rt < NRT; ++rt)
        Qd::st(sF + (16 * rt + c) * LDD + 16 * w + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(acc[rt]));
      __syncthreads();
    }
    // raw erase logits into region X (the fold is done with the state)
    CARVE_STAGE_ROWS(sBx, cbx, false);
    // the previous block's outputs
    if (oprev >= 0) {
      int cs = c, gs = g;
      asm volatile("" : "+v"(cs), "+v"(gs));
      for (int bb = 0; bb < NB; ++bb) Qd::st(o + (oprev + 16 * bb + cs) * rs + 16 * w + 4 * gs, oq[bb]);
    }

    // ---- tau^T[r][t] = tanh(F[r] . q_t) -> sTau[t][r] ---------------------------
    if constexpr (NW % NRT == 0) {
      // every tile of this wave has the same fold rows: read them once
      const int rt = w % NRT;
      quad fq[D / 16];
      for (int jp = 0; jp < D / 32; ++jp) {
        const T* fr = sF + (16 * rt + c) * LDD + 32 * jp + ((4 * g) ^ CARVE_QX(c));
        fq[2 * jp] = Qd::ld(fr);
        fq[2 * jp + 1] = Qd::ld(fr + 16);
      }
      for (int bb = w / NRT; bb < NB; bb += NW / NRT) {
        f32x4 acc = zero4();
        for (int jp = 0; jp < D / 32; ++jp) {
          const T* qr = sQ + (16 * bb + c) * LDD + 32 * jp + ((4 * g) ^ CARVE_QX(c));
          acc = Qd::mma32(fq[2 * jp], fq[2 * jp + 1], Qd::ld(qr), Qd::ld(qr + 16), acc);
        }
        for (int e = 0; e < 4; ++e) acc[e] = tanh_f(acc[e]);
        Qd::st(sTau + (16 * bb + c) * LDR + 16 * rt + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(acc));
      }
    } else {
      for (int x = w; x < NRT * NB; x += NW) {
        const int rt = x % NRT, bb = x / NRT;
        f32x4 acc = zero4();
        for (int jp = 0; jp < D / 32; ++jp) {
          const T* fr = sF + (16 * rt + c) * LDD + 32 * jp + ((4 * g) ^ CARVE_QX(c));
          const T* qr = sQ + (16 * bb + c) * LDD + 32 * jp + ((4 * g) ^ CARVE_QX(c));
          acc = Qd::mma32(Qd::ld(fr), Qd::ld(fr + 16), Qd::ld(qr), Qd::ld(qr + 16), acc);
        }
        for (int e = 0; e < 4; ++e) acc[e] = tanh_f(acc[e]);
        Qd::st(sTau + (16 * bb + c) * LDR + 16 * rt + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(acc));
      }
    }
    __syncthreads();

    // ---- gates ------------------------------------------------------------------
    // key side, key tile w: lane (g, c) of tile bb holds token 16 bb + c and keys
    // j = 16 w + 4 g + e; prefix sums run along the 16 lanes of a row.  Log
    // retentions are kept in units of log 2 here (lam below is lam / log 2), so
    // that every exponential of this step is one exp2.
    f32x4 lam[NB];
    {
      f32x4 carry = zero4();
      for (int bb = 0; bb < NB; ++bb) {
        f32x4 z = zero4();
        for (int ks = 0; ks < NRB; ++ks)
          z = Qd::mma16(fVb[ks], Qd::ld(sTau + (16 * bb + c) * LDR + 16 * ks + ((4 * g) ^ CARVE_QX(c))), z);
        const f32x4 bxv = Qd::f32(Qd::ld(sBx + (16 * bb + c) * LDD + 16 * w + ((4 * g) ^ CARVE_QX(c))));
        f32x4 gv;
        if constexpr (GATED) {
          const f32x4 fv = Qd::f32(pf[bb]);
          const f32x4 na = *reinterpret_cast<const f32x4*>(sGate + 16 * w + 4 * g);
          const f32x4 tf = *reinterpret_cast<const f32x4*>(sGate + D + 16 * w + 4 * g);
          for (int e = 0; e < 4; ++e) gv[e] = na[e] * softplus2_f(fv[e] + tf[e]);   // g / log 2
        } else {
          gv = pg[bb];
        }
        for (int e = 0; e < 4; ++e) {
          const float sp = softplus2_f(z[e] + bxv[e]);
          const float ell = GATED ? gv[e] - sp : fmaf(gv[e], kLog2e, -sp);
          lam[bb][e] = bb == 0 ? row_scan(ell) : carry[e] + row_scan(ell);
          carry[e] = row_bcast15(lam[bb][e]);
        }
      }
    }
    // lam at the end of tile i, c_i, is lane 15 of the row (row_bcast15).  A key
    // channel whose block retention falls below e^{-kWideLog} takes per-tile
    // references; the wave's vote goes to LDS for the products after the next
    // barrier.
    {
      bool wch[4];
      bool mine = false;
      for (int e = 0; e < 4; ++e) {
        wch[e] = NB > 1 && row_bcast15(lam[NB - 1][e]) < -kWideLog * kLog2e;
        mine = mine || wch[e];
      }
      const bool wave_wide = __any(mine) != 0;
      if (NB > 1 && lane == 0) sFlag[w] = wave_wide ? 1 : 0;
      f32x4 fill, cprev = zero4();   // e^{lam_{t-1} - m} for the first token of tile bb; c_{bb-1}
      // factor tables: lane c of the row forms row c for the row's 4 channels
      // (one reference: e^{rho} in rows St, Up; 1 in Half, Gap; e^{lam_end} in End).
      // Row c as a linear form in the tile ends: exponent sum_i tc[i] c_i on
      // per-tile references, tn lam_end on one reference.  The lane index is
      // taken opaque here so that no lane mask is hoisted out of the blocks.
      float tc[NB], tn = 0.0f;
      {
        int cr = c;
        asm volatile("" : "+v"(cr));
        for (int i = 0; i < NB; ++i) tc[i] = 0.0f;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const float h = (cr == kTabSt + i) ? 0.5f : 0.0f;     // m_i = (c_{i-1} + c_i) / 2
          const float u = (cr == kTabUp + i) ? 0.5f : 0.0f;     // lam_end - m_i
          const float f = (cr == kTabHalf + i) ? 0.5f : 0.0f;   // c_i - m_i
          tc[i] += h - u + f;
          if (i > 0) tc[i - 1] += h - u - f;
          tc[NB - 1] += 2.0f * u;
          tn += h + u;
#pragma unroll
          for (int j = 0; j + 2 <= i; ++j) {
            const float q = (cr == kTabGap + (i - 2) * (i - 1) / 2 + j) ? 0.5f : 0.0f;   // m_i - c_j
            tc[i] += q;
            tc[i - 1] += q;
            tc[j] -= 2.0f * q;
          }
        }
        if (cr == kTabEnd) {
          tc[NB - 1] += 1.0f;
          tn = 1.0f;
        }
      }
      f32x4 x;
      for (int e = 0; e < 4; ++e) {
        const float lend = row_bcast15(lam[NB - 1][e]);
        float xe = tn * lend;
        if (wave_wide) {
          // (the per-tile forms only where a channel of this wave needs them)
          float xw = 0.0f;
          for (int i = 0; i < NB; ++i) xw = fmaf(tc[i], row_bcast15(lam[i][e]), xw);
          xe = wch[e] ? xw : xe;
        }
        x[e] = exp2_f(xe);
        fill[e] = exp2_f(-0.5f * lend);
      }
      if (c < NTAB) *reinterpret_cast<f32x4*>(sTab + c * D + 16 * w + 4 * g) = x;
      // decayed operands of the key tile: Kt = k e^{lam_{t-1} - m}, Qt = q e^{lam - m},
      // Ki = k e^{m - lam} (each one exp2 of the scaled exponents); PER_CHANNEL_:
      // the channels flagged in wch take per-tile references (the branch is
      // taken by waves with such a channel)
#define CARVE_GATE_OPERANDS(PER_CHANNEL_)                                                          \
  for (int bb = 0; bb < NB; ++bb) {                                                                \
    T* kp = sKi + (16 * bb + c) * LDD + 16 * w + ((4 * g) ^ CARVE_QX(c));                          \
    const f32x4 kv = Qd::f32(Qd::ld(kp));                                                          \
    T* qp = sQ + (16 * bb + c) * LDD + 16 * w + ((4 * g) ^ CARVE_QX(c));                           \
    const f32x4 qv = Qd::f32(Qd::ld(qp));                                                          \
    f32x4 kt, qt, ki;                                                                              \
    for (int e = 0; e < 4; ++e) {                                                                  \
      float m = 0.5f * row_bcast15(lam[NB - 1][e]), f0 = fill[e];                                   \
      if (PER_CHANNEL_) {                                                                          \
        /* per-tile reference: e^{c_{bb-1} - m} = e^{m - c_bb} */                                  \
        const float ce = row_bcast15(lam[bb][e]);                                                  \
        const float mt = 0.5f * (cprev[e] + ce);                                                   \
        const float eb = row_bcast15(exp2_f(mt - lam[bb][e]));                                      \
        m = wch[e] ? mt : m;                                                                       \
        f0 = wch[e] ? eb : f0;                                                                     \
        cprev[e] = ce;                                                                             \
      }                                                                                            \
      float E, Ei;                                                                                 \
      exp2_pm(lam[bb][e] - m, E, Ei);                                                              \
      kt[e] = kv[e] * row_shr1(E, f0);                                                             \
      qt[e] = qv[e] * E;                                                                           \
      ki[e] = kv[e] * Ei;                                                                          \
      fill[e] = row_bcast15(E); /* one reference: E of the tile's last token */                    \
    }                                                                                              \
    Qd::st(sKt + (16 * bb + c) * LDD + 16 * w + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(kt));             \
    Qd::st(qp, Qd::cvt(qt));                                                                       \
    Qd::st(kp, Qd::cvt(ki));                                                                       \
  }
      if (wave_wide) {
        CARVE_GATE_OPERANDS(true)
      } else {
        CARVE_GATE_OPERANDS(false)
      }
#undef CARVE_GATE_OPERANDS
    }
    // value side, value tile w: rows t = 16 bb + 4 g + e, column v = 16 w + c.
    // The operand quads are taken here (the staged rows share LDS with the
    // coupling tiles); the write gate w and w * v are formed after the barrier,
    // at the start of the coupling step: the gate step is bound by the SIMDs'
    // VALU issue, the coupling step by its matrix-core and LDS chains.
    quad vqs[NB], wxqs[NB];
    for (int bb = 0; bb < NB; ++bb) {
      quad vq = pv[bb], wxq;
      if constexpr (!SW) wxq = pwx[bb];
      if constexpr (SVW) {
        // row t = 16 bb + c, elements 16 w + 4 g .. + 3 of the swizzled tiles
        const int by = (16 * w + 4 * g) * (int)sizeof(T), t = 16 * bb + c;
        const T* r0 = sVW + t * D + ((((by >> 4) ^ (t & (NC - 1))) << 4) | (by & 15)) / (int)sizeof(T);
        vq = Qd::ld(r0);
        if constexpr (!SW) wxq = Qd::ld(r0 + WB * D);
      } else if constexpr (ACT) {
        vq = Qd::cvt(silu4(Qd::f32(vq)));
      }
      vqs[bb] = vq;
      if constexpr (!SW) wxqs[bb] = wxq;
    }
    {
      const int nx = blk + 1 < nblk ? blk + 1 : blk;
      CARVE_PREFETCH_GATES(nx);
    }
    __syncthreads();

    // ---- coupling tiles, diagonal inverses, state products ---------------------
    bool wide = false;   // some key channel of the block on per-tile references
    if constexpr (NB > 1) {
      int f = 0;
      for (int x = 0; x < NW; ++x) f |= sFlag[x];
      wide = __builtin_amdgcn_readfirstlane(f) != 0;
    }
    // w * v of each tile (the write gate from tau_w Vw^T + wx, or the token's
    // scalar gate)
    f32x4 wv[NB];
    for (int bb = 0; bb < NB; ++bb) {
      const f32x4 vv = Qd::mma16(vqs[bb], fI, zero4());
      if constexpr (SW) {
        const f32x4 ws = *reinterpret_cast<const f32x4*>(sWs + par * WB + 16 * bb + 4 * g);
        for (int e = 0; e < 4; ++e) wv[bb][e] = ws[e] * vv[e];
      } else {
        f32x4 z = zero4();
        for (int ks = 0; ks < NRB; ++ks)
          z = Qd::mma16(Qd::ld(sTau + (16 * bb + c) * LDR + RP + 16 * ks + ((4 * g) ^ CARVE_QX(c))), fVw[ks], z);
        z = Qd::mma16(wxqs[bb], fI, z);                // + wx, moved into this layout
        for (int e = 0; e < 4; ++e) wv[bb][e] = sigmoid_f(z[e]) * vv[e];
      }
    }
    if (!(kSplitRoles && w < NOW)) CARVE_STORE_S(NJT / 2, NJT);
    CARVE_PREFETCH_G(blk + 1 < nblk ? blk + 1 : blk);
    const float* bcur = sBeta + par * WB;
    // Diagonal 16 x 16 tiles: T_ii = (I + A_ii)^{-1}.  A_ii is strictly lower
    // triangular, so with M = -A_ii (M^16 = 0)
    //   T_ii = sum_{k < 16} M^k = (I + M)(I + M^2)(I + M^4)(I + M^8):
    // eight f32 matrix-core products (M^2, M^4 and their transposes, M^8, then
    // the three factors), no serial substitution.  An operand used on the left
    // is held as its transpose in the result layout, so each power is formed
    // both ways.  NDW waves (one per SIMD) take the diagonal tiles, the others
    // (all waves when each has a diagonal tile) the off-diagonal ones.
    // The off-diagonal workers carry the step's longest chains: they take issue
    // priority over the diagonal-inverse wave on their SIMD until the barrier.
    if (kSplitRoles && w < NOW) __builtin_amdgcn_s_setprio(2);
    if (w >= NW - NDW) {
      typedef Quad<float> Qf;
      for (int i = NW - 1 - w; i < NB; i += NDW) {
        f32x4 acc = zero4(), accT = zero4();
        const T* kr = sKt + (16 * i + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        const T* ir = sKi + (16 * i + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        for (int jp = 0; jp < D / 32; ++jp) {
          const quad k0 = Qd::ld(kr + 32 * jp), k1 = Qd::ld(kr + 32 * jp + 16);
          const quad i0 = Qd::ld(ir + 32 * jp), i1 = Qd::ld(ir + 32 * jp + 16);
          acc = Qd::mma32(k0, k1, i0, i1, acc);     // Kt_{t = 16 i + 4 g + e} . Ki_{s = 16 i + c}
          accT = Qd::mma32(i0, i1, k0, k1, accT);   // Ki_{s = 16 i + 4 g + e} . Kt_{t = 16 i + c}
        }
        const f32x4 bt = *reinterpret_cast<const f32x4*>(bcur + 16 * i + 4 * g);
        const float bc = bcur[16 * i + c];
        f32x4 mB, mA, I4;   // M in the result layout (M[4g+e][c]) and transposed (M[c][4g+e])
        for (int e = 0; e < 4; ++e) {
          mB[e] = (c < 4 * g + e) ? -bt[e] * acc[e] : 0.0f;
          mA[e] = (4 * g + e < c) ? -bc * accT[e] : 0.0f;
          I4[e] = (4 * g + e == c) ? 1.0f : 0.0f;
        }
        const f32x4 M2 = Qf::mma16(mA, mB, zero4());
        const f32x4 M2t = Qf::mma16(mB, mA, zero4());
        const f32x4 M4 = Qf::mma16(M2t, M2, zero4());
        const f32x4 M4t = Qf::mma16(M2, M2t, zero4());
        const f32x4 M8 = Qf::mma16(M4t, M4, zero4());
        const f32x4 W = Qf::mma16(M4t + I4, M8 + I4, zero4());   // (I + M^4)(I + M^8)
        const f32x4 W2 = Qf::mma16(M2t + I4, W, zero4());        // (I + M^2) W
        const f32x4 Ti = Qf::mma16(mA + I4, W2, zero4());        // (I + M) W2
        // T_ii[t = 4g + e][s = c] at (s, t) of sTmT
        Qd::st(sTmT + (i * 16 + c) * LDB + ((4 * g) ^ CARVE_QX(c)), Qd::cvt(Ti));
      }
    }
    if (NOW == NW || w < NOW) {
      // off-diagonal tiles of -A and all tiles of P, stored [t][s]; a scalar
      // loop over this wave's tiles (addresses from opaque lane coordinates)
      int ct = c, gt = g;
      asm volatile("" : "+v"(ct), "+v"(gt));
#pragma unroll 1
      for (int x = w; x < NTA + NTP; x += NOW) {
        const bool isA = x < NTA;
        const int y = isA ? x : x - NTA;
        const int i = tri_row(y, isA), j = tri_col(y, isA);
        // acc[e] = Ki_{s = 16 j + 4 g + e} . X_{t = 16 i + c}, X = Kt (A) or Qt (P)
        const T* ar = sKi + (16 * j + ct) * LDD + ((4 * gt) ^ CARVE_QX(ct));
        const T* br = (isA ? sKt : sQ) + (16 * i + ct) * LDD + ((4 * gt) ^ CARVE_QX(ct));
        f32x4 acc = zero4();
        if (wide && i > j) {
          // per-tile references: Ki e^{c_j - m_j} against X e^{m_i - c_j}; lane
          // quads hold channels 32 jp + 4 g .. + 3 and 16 further
          const float* fa = sTab + (kTabHalf + j) * D + 4 * gt;
          const float* fb = sTab + (i == j + 1 ? kTabHalf + i : kTabGap + (i - 2) * (i - 1) / 2 + j) * D + 4 * gt;
          for (int jp = 0; jp < D / 32; ++jp) {
            const quad a0 = scale_q<T>(Qd::ld(ar + 32 * jp), fa + 32 * jp);
            const quad a1 = scale_q<T>(Qd::ld(ar + 32 * jp + 16), fa + 32 * jp + 16);
            const quad b0 = scale_q<T>(Qd::ld(br + 32 * jp), fb + 32 * jp);
            const quad b1 = scale_q<T>(Qd::ld(br + 32 * jp + 16), fb + 32 * jp + 16);
            acc = Qd::mma32(a0, a1, b0, b1, acc);
          }
        } else {
          for (int jp = 0; jp < D / 32; ++jp)
            acc = Qd::mma32(Qd::ld(ar + 32 * jp), Qd::ld(ar + 32 * jp + 16), Qd::ld(br + 32 * jp),
                            Qd::ld(br + 32 * jp + 16), acc);
        }
        f32x4 val;
        if (isA) {
          const float bt = bcur[16 * i + ct];
          for (int e = 0; e < 4; ++e) val[e] = -bt * acc[e];
          Qd::st(sA + (16 * i + ct) * LDW + 16 * j + ((4 * gt) ^ CARVE_QX(ct)), Qd::cvt(val));
        } else {
          for (int e = 0; e < 4; ++e) val[e] = (i > j || 4 * gt + e <= ct) ? acc[e] : 0.0f;
          Qd::st(sP + (16 * i + ct) * LDW + 16 * j + ((4 * gt) ^ CARVE_QX(ct)), Qd::cvt(val));
        }
      }
    }
    // on the value tile (rows t = 16 bb + 4 g + e, column v): XQ = Qt S^T and the
    // right-hand side R = beta (w * v - Kt S^T)
    f32x4 RH[NB], XQ[NB];
    if (!wide) {
      quad sb[NJT];   // S diag(e^{rho}) as the B operand
      for (int jt = 0; jt < NJT; ++jt)
        sb[jt] = Qd::cvt(St[jt] * *reinterpret_cast<const f32x4*>(sTab + kTabSt * D + 16 * jt + 4 * g));
      for (int bb = 0; bb < NB; ++bb) {
        f32x4 xk = zero4();
        XQ[bb] = zero4();
        const T* kr = sKt + (16 * bb + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        const T* qr = sQ + (16 * bb + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        for (int jp = 0; jp < NJT / 2; ++jp) {
          xk = Qd::mma32(Qd::ld(kr + 32 * jp), Qd::ld(kr + 32 * jp + 16), sb[2 * jp], sb[2 * jp + 1], xk);
          XQ[bb] = Qd::mma32(Qd::ld(qr + 32 * jp), Qd::ld(qr + 32 * jp + 16), sb[2 * jp], sb[2 * jp + 1], XQ[bb]);
        }
        const f32x4 bt = *reinterpret_cast<const f32x4*>(bcur + 16 * bb + 4 * g);
        for (int e = 0; e < 4; ++e) RH[bb][e] = bt[e] * (wv[bb][e] - xk[e]);
      }
    } else {
      // S diag(e^{m_bb}) formed per tile, two state columns at a time
      for (int bb = 0; bb < NB; ++bb) {
        f32x4 xk = zero4();
        XQ[bb] = zero4();
        const T* kr = sKt + (16 * bb + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        const T* qr = sQ + (16 * bb + c) * LDD + ((4 * g) ^ CARVE_QX(c));
        const float* fs = sTab + (kTabSt + bb) * D + 4 * g;
        for (int jp = 0; jp < NJT / 2; ++jp) {
          const quad s0 = Qd::cvt(St[2 * jp] * *reinterpret_cast<const f32x4*>(fs + 32 * jp));
          const quad s1 = Qd::cvt(St[2 * jp + 1] * *reinterpret_cast<const f32x4*>(fs + 32 * jp + 16));
          xk = Qd::mma32(Qd::ld(kr + 32 * jp), Qd::ld(kr + 32 * jp + 16), s0, s1, xk);
          XQ[bb] = Qd::mma32(Qd::ld(qr + 32 * jp), Qd::ld(qr + 32 * jp + 16), s0, s1, XQ[bb]);
        }
        const f32x4 bt = *reinterpret_cast<const f32x4*>(bcur + 16 * bb + 4 * g);
        for (int e = 0; e < 4; ++e) RH[bb][e] = bt[e] * (wv[bb][e] - xk[e]);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();

    // ---- value tile: blocked substitution for u, outputs, state carry ---------------
    CARVE_PREFETCH_VW(blk + 1 < nblk ? blk + 1 : blk);
    quad uq[NB];
    for (int i = 0; i < NB; ++i) {
      f32x4 r = RH[i];
      for (int j = 0; j < i; ++j) r = Qd::mma16(Qd::ld(sA + (16 * i + c) * LDW + 16 * j + ((4 * g) ^ CARVE_QX(c))), uq[j], r);
      const f32x4 u = Qd::mma16(Qd::ld_tr_sw(sTmT + i * 16 * LDB, LDB, 0, 0, g, c), Qd::cvt(r), zero4());
      uq[i] = Qd::cvt(u);
      f32x4 O = XQ[i];
      for (int j = 0; j <= i; ++j) O = Qd::mma16(Qd::ld(sP + (16 * i + c) * LDW + 16 * j + ((4 * g) ^ CARVE_QX(c))), uq[j], O);
      oq[i] = Qd::cvt(Qd::mma16(Qd::cvt(O), fI, zero4()));
    }
    if (!wide) {
      // S <- (S e^{rho} + u^T Ki) e^{rho}, rho = lam_end / 2
      for (int jt = 0; jt < NJT; ++jt) {
        const f32x4 er = *reinterpret_cast<const f32x4*>(sTab + kTabSt * D + 16 * jt + 4 * g);
        f32x4 acc = St[jt] * er;
        for (int kp = 0; kp < NB / 2; ++kp)
          acc = Qd::mma32(Qd::ld_tr_sw(sKi, LDD, 32 * kp, 16 * jt, g, c), Qd::ld_tr_sw(sKi, LDD, 32 * kp + 16, 16 * jt, g, c),
                          uq[2 * kp], uq[2 * kp + 1], acc);
        if (NB & 1) acc = Qd::mma16(Qd::ld_tr_sw(sKi, LDD, 16 * (NB - 1), 16 * jt, g, c), uq[NB - 1], acc);
        St[jt] = acc * er;
      }
    } else {
      // S <- S e^{lam_end} + u^T (Ki_s e^{lam_end - m_j}) (the transposed Ki quads
      // hold one channel, 16 jt + c, and four tokens of tile j)
      for (int jt = 0; jt < NJT; ++jt) {
        f32x4 acc = St[jt] * *reinterpret_cast<const f32x4*>(sTab + kTabEnd * D + 16 * jt + 4 * g);
        for (int kp = 0; kp < NB / 2; ++kp) {
          const quad k0 = Qd::cvt(Qd::f32(Qd::ld_tr_sw(sKi, LDD, 32 * kp, 16 * jt, g, c)) *
                                  sTab[(kTabUp + 2 * kp) * D + 16 * jt + c]);
          const quad k1 = Qd::cvt(Qd::f32(Qd::ld_tr_sw(sKi, LDD, 32 * kp + 16, 16 * jt, g, c)) *
                                  sTab[(kTabUp + 2 * kp + 1) * D + 16 * jt + c]);
          acc = Qd::mma32(k0, k1, uq[2 * kp], uq[2 * kp + 1], acc);
        }
        if (NB & 1) {
          const quad k0 = Qd::cvt(Qd::f32(Qd::ld_tr_sw(sKi, LDD, 16 * (NB - 1), 16 * jt, g, c)) *
                                  sTab[(kTabUp + NB - 1) * D + 16 * jt + c]);
          acc = Qd::mma16(k0, uq[NB - 1], acc);
        }
        St[jt] = acc;
      }
    }
    oprev = t0;
  }
  for (int bb = 0; bb < NB; ++bb) Qd::st(o + (oprev + 16 * bb + c) * rs + 16 * w + 4 * g, oq[bb]);
  if (a.S_T) {
    float* dst = a.S_T + soff + (16 * w + c) * D + 4 * g;
    for (int jt = 0; jt < NJT; ++jt) *reinterpret_cast<f32x4*>(dst + 16 * jt) = St[jt];
  }
#undef CARVE_PREFETCH_Q
#undef CARVE_PREFETCH_GATES
#undef CARVE_PREFETCH_G
#undef CARVE_PREFETCH_VW
#undef CARVE_STORE_S
#undef CARVE_STAGE_VW
#undef CARVE_STAGE_ROWS
#undef CARVE_QX
}

// ---------------------------------------------------------------------------
// host-side launch (one variant)
// ---------------------------------------------------------------------------
template <typename T, int D, int WB, int RP, int VAR>
static int launch_chain_t(const FwdArgs& a, hipStream_t stream) {
  constexpr ChainLds lay = chain_lds<T, D, WB, RP, VAR>();
  if constexpr (lay.total > kMaxLdsBytes) {
    (void)a;
    (void)stream;
    return CARVE_ERR_UNSUPPORTED;
  } else {
  auto kern = carve_chain_fwd_kernel<T, D, WB, RP, VAR>;
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
}

template <typename T, int D, int RP, int VAR>
static int launch_chain_w(const FwdArgs& a, int WB, hipStream_t s) {
  if (WB == 16) return launch_chain_t<T, D, 16, RP, VAR>(a, s);
  if (WB == 32) return launch_chain_t<T, D, 32, RP, VAR>(a, s);
  if (WB == 64) return launch_chain_t<T, D, 64, RP, VAR>(a, s);
  return CARVE_ERR_UNSUPPORTED;
}

template <typename T, int VAR>
static int launch_chain_d(const FwdArgs& a, int D, int WB, hipStream_t s) {
  if (a.RP == 32) {
    if (D == 32) return launch_chain_w<T, 32, 32, VAR>(a, WB, s);
    if (D == 64) return launch_chain_w<T, 64, 32, VAR>(a, WB, s);
    if (D == 128) return launch_chain_w<T, 128, 32, VAR>(a, WB, s);
  } else if (a.RP == 64) {
    if (D == 32) return launch_chain_w<T, 32, 64, VAR>(a, WB, s);
    if (D == 64) return launch_chain_w<T, 64, 64, VAR>(a, WB, s);
    if (D == 128) return launch_chain_w<T, 128, 64, VAR>(a, WB, s);
  }
  return CARVE_ERR_UNSUPPORTED;
}

template <int VAR>
int launch_chain_fwd_var(const FwdArgs& a, int dtype, int D, int WB, hipStream_t s) {
  if (dtype == CARVE_BF16) return launch_chain_d<bf16_t, VAR>(a, D, WB, s);
  return launch_chain_d<float, VAR>(a, D, WB, s);
}

}  // namespace carve
