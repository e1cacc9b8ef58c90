// carve_rec.h -- chunk recompute of the CARVE backward on gfx950.
//
// rec_chunk() recomputes one gate chunk of one (batch, head) from its start
// state (S_chunks, written by the forward) and writes the chunk record that the
// adjoint reads (ChunkRec): the fold F, tau, and T, P and the scaled start
// state of every 16-token WY block, and (except with the decay formed in the
// kernels) the retention factors E and the erase gate of every token.  Every chunk is independent, so the
// recompute is chunk-parallel.  Wave w of the workgroup owns the 16-wide tile w
// of the value axis and the 16-wide tile w of the key axis:
//   * the state lives in registers as S^T tiles (rows = key index j, columns =
//     the wave's 16 value rows v), in the matrix-core result layout;
//   * everything on the value side (predictions, WY solve, state update) is
//     wave-local, so the token-serial part of a sub-chunk runs without barriers;
//   * the key-side gate arithmetic (erase gate, log retention, its prefix sums
//     and the decayed keys/queries) runs on the wave's key tile.
//
// Per gate chunk with start state S_hat (Eq. content_readout):
//   F = [Ub; Uw] S_hat                         (fold, once per chunk)
//   tau = tanh(q F^T), z_b = bx + tau_b Vb^T, z_w = wx + tau_w Vw^T
//   l = g - softplus(z_b) = log(exp(g) (1 - b)), w = sigmoid(z_w)
// and then, for consecutive 16-token blocks (the WY form of Sec. 6.2 applied
// block by block; every block of the chunk uses the same F), with lam = prefix
// sums of l inside the block (lam_{-1} = 0), the block reference
// rho = lam_15 / 2 per key channel (the middle of the block's log-retention
// range), state S at the block start and u the WY "pseudo values":
//   Kt_t = k_t e^{lam_{t-1} - rho},  Ki_s = k_s e^{rho - lam_s},  Qt_t = q_t e^{lam_t - rho}
//   S' = S diag(e^{rho})
//   A_ts = beta_t Kt_t . Ki_s (s < t),  P_ts = Qt_t . Ki_s (s <= t)
//   T = (I + A)^{-1},  R_t = beta_t (w_t * v_t - S' Kt_t),  u = T R
//   S <- (S' + sum_s u_s Ki_s^T) diag(e^{lam_15 - rho})    (e^{lam_15 - rho} = e^{rho})
// which is the recurrence of Eq. carve_state rewritten exactly (every pair of
// factors multiplies to e^{lam_a - lam_b} with a >= b).  No factor exceeds
// e^{|lam_15| / 2}.  The record keeps, per block, T, P and the scaled start
// state S' (the adjoint evaluates the block with the same reference).
//
// With the scalar write gate (kVarScalarW) F = Ub S_hat has R rows and
// w_t = sigmoid(wx_t) is one scalar per token and head, staged with beta.
// With the input activations (kVarAct) q, k, v arrive raw: q rows are staged
// as SiLU(raw) / |SiLU(raw)|; a key's norm is summed from per-wave partials
// through LDS (each wave holds 16 of its channels); v is SiLU(raw).
//
// Precondition (not checked): within any 16-token block the log retention
// summed over the block stays above about -170 per key channel, so that
// e^{|block log retention| / 2} is finite in f32 and bf16.
#pragma once
#include "carve_kernels.h"

namespace carve {

// One chunk ch0 of (batch, head) bh; LW-token sub-chunks (LW | L).  smem is the
// workgroup's dynamic LDS (RecLds layout).  Ends with a workgroup barrier, so
// the caller may reuse the LDS at once; the record stores may still be in
// flight.
// GATED: g is formed from its raw logit f as -exp(A) softplus(f + tau_f)
// (Eq. decay_gate), A and tau_f of the head held in LDS.
template <typename T, int D, int LW, int RP, int VAR>
__device__ __forceinline__ void rec_chunk(const FwdArgs& a, const int bh, const int ch0, char* smem) {
  typedef Quad<T> Qd;
  typedef typename Qd::q quad;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr bool GATED = (VAR & kVarGated) != 0;
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr bool ACT = (VAR & kVarAct) != 0;
  constexpr int NT = fwd_threads(D);
  constexpr int NW = NT / 64;          // waves == 16-wide tiles of the key / value axis
  constexpr int NJT = D / 16;
  constexpr int NB = LW / 16;          // 16-token blocks per sub-chunk
  constexpr int R2 = fold_rows(RP, VAR);
  constexpr int NRT = R2 / 16;         // 16-row tiles of the fold operand ([Ub; Uw] or Ub) and of F
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDD = D + PAD, LDR = R2 + PAD, LDB = 16 + PAD;
  constexpr int VEC = 16 / sizeof(T);          // token elements per 16-byte vector
  constexpr int NVQ = LW * D / VEC;            // 16-byte vectors of a q tile
  constexpr int NQV = (NVQ + NT - 1) / NT;     // per thread
  static_assert(NW == NJT, "one wave per 16-wide tile");
  static_assert(D % 32 == 0, "K32 steps over the key / value axis");
  static_assert(NVQ % 64 == 0, "whole waves of row chunks (the row sums run over lanes)");

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int H = a.H, Tn = a.T, L = a.L, R = a.R;
  const int nch = Tn / L, msub = L / LW;
  const int b = bh / H, h = bh % H;

  constexpr RecLds lay = rec_lds<T, D, LW, RP, VAR>();
  T* sU = reinterpret_cast<T*>(smem + lay.U);      // [R2][LDD]   [Ub; 0; Uw; 0] or [Ub; 0]
  T* sQ = reinterpret_cast<T*>(smem + lay.Q);      // [LW][LDD]   raw q
  T* sF = reinterpret_cast<T*>(smem + lay.F);      // [R2][LDD]   F
  T* sTau = reinterpret_cast<T*>(smem + lay.Tau);  // [LW][LDR]   tau (b half | w half)
  float* sBeta = reinterpret_cast<float*>(smem + lay.Beta);   // [LW] beta, then [LW] sigmoid(wx) (SW)
  T* sS = reinterpret_cast<T*>(smem + lay.S);      // [D][LDD]    S_hat[v][j] (chunk start)
  T* sKt = reinterpret_cast<T*>(smem + lay.Kt);    // [LW][LDD]
  T* sQt = reinterpret_cast<T*>(smem + lay.Qt);    // [LW][LDD]
  T* sKi = reinterpret_cast<T*>(smem + lay.Ki);    // [LW][LDD]
  float* sGam = reinterpret_cast<float*>(smem + lay.Gam);  // [NB][D]     e^{rho} = e^{lam_15 / 2}
  float* sAT = reinterpret_cast<float*>(smem + lay.AT);    // [NB][16][20] A^T per block
  T* sTm = reinterpret_cast<T*>(smem + lay.Tm);            // [NB][16][LDB] T per block
  float* sGate = reinterpret_cast<float*>(smem + lay.Gate);  // [2][D] -exp(A), tau_f (GATED)
  float* sKn = reinterpret_cast<float*>(smem + lay.Kn);      // [NW][LW] partial |SiLU(k)|^2 (ACT)

  // token tensors addressed from this (batch, head)'s first element with 32-bit
  // offsets t * rs + column (rs = H * D elements between consecutive tokens)
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
    sU[rr * LDD + i] = (T)u;
  }
  // Vb / Vw as constant operand quads: lane (g, c) holds V[16 w + c][16 ks + 4 g + e]
  quad fVb[RP / 16], fVw[RP / 16];
  for (int ks = 0; ks < RP / 16; ++ks) {
    f32x4 tb, tw;
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * ks + 4 * g + e;
      tb[e] = r < R ? a.Vb[(16 * w + c) * R + r] : 0.0f;
      tw[e] = (!SW && r < R) ? a.Vw[(16 * w + c) * R + r] : 0.0f;
    }
    fVb[ks] = Qd::cvt(tb);
    fVw[ks] = Qd::cvt(tw);
  }
  // identity operand: lane (g, c) holds I[4 g + e][c]
  quad fI;
  {
    f32x4 t;
    for (int e = 0; e < 4; ++e) t[e] = (4 * g + e == c) ? 1.0f : 0.0f;
    fI = Qd::cvt(t);
  }

  // ---- state: St[jt][i] = S[v = 16 w + c][j = 16 jt + 4 g + i] ---------------
  f32x4 St[NJT];
  {
    const float* src = a.S_chunks + ((size_t)bh * nch + ch0) * D * D + (16 * w + c) * D + 4 * g;
    for (int jt = 0; jt < NJT; ++jt) St[jt] = gload4(src + 16 * jt);
  }
  const ChunkRec cr = chunk_rec(sizeof(T), D, L, R2);
  char* rec = reinterpret_cast<char*>(a.rec) + ((size_t)bh * nch + ch0) * cr.total;

  // ---- prefetch registers for the next sub-chunk ------------------------------
  u32x4 pq[NQV];
  T pbeta = (T)0.0f, pws = (T)0.0f;   // beta and (SW) the write logit of token tid
  quad pbx[NB], pk[NB], pwx[NB], pv[NB];
  f32x4 pg[NB];     // g per tile (ungated)
  quad pf[NB];      // f per tile (GATED)
#define CARVE_REC_PREFETCH_Q(TILE_)                                                     \
  do {                                                                                  \
    const int tt0_ = (TILE_) * LW;                                                      \
    for (int u_ = 0; u_ < NQV; ++u_) {                                                  \
      const int x_ = tid + u_ * NT;                                                     \
      if (NVQ % NT != 0 && x_ >= NVQ) break;                                            \
      const int t_ = x_ / (D / VEC), j_ = (x_ % (D / VEC)) * VEC;                       \
      pq[u_] = *reinterpret_cast<const u32x4*>(q + (tt0_ + t_) * rs + j_);              \
    }                                                                                   \
    if (tid < LW) {                                                                     \
      pbeta = beta[(tt0_ + tid) * H];                                                   \
      if constexpr (SW) pws = wx[(tt0_ + tid) * H];                                     \
    }                                                                                   \
  } while (0)
#define CARVE_REC_PREFETCH_GATES(TILE_)                                                 \
  do {                                                                                  \
    const int tt0_ = (TILE_) * LW;                                                      \
    for (int bb_ = 0; bb_ < NB; ++bb_) {                                                \
      const int e_ = (tt0_ + 16 * bb_ + c) * rs + 16 * w + 4 * g;                       \
      pbx[bb_] = Qd::ld(bx + e_);                                                       \
      pk[bb_] = Qd::ld(k + e_);                                                         \
      if constexpr (!SW) pwx[bb_] = Qd::ld(wx + e_);                                    \
      pv[bb_] = Qd::ld(v + e_);                                                         \
      if constexpr (GATED) pf[bb_] = Qd::ld(fl + e_);                                   \
      else pg[bb_] = *reinterpret_cast<const f32x4*>(gl + e_);                          \
    }                                                                                   \
  } while (0)
  const int tile0 = ch0 * msub, ntiles = tile0 + msub;
  CARVE_REC_PREFETCH_Q(tile0);
  CARVE_REC_PREFETCH_GATES(tile0);

  for (int m = 0; m < msub; ++m) {
    const int tile = tile0 + m;

    // ---- P0: stage q and beta; chunk start state --------------------------------
    if (m == 0)
      for (int jt = 0; jt < NJT; ++jt) Qd::st(sS + (16 * w + c) * LDD + 16 * jt + 4 * g, Qd::cvt(St[jt]));
    for (int u = 0; u < NQV; ++u) {
      const int x = tid + u * NT;
      if (NVQ % NT != 0 && x >= NVQ) break;
      const int t = x / (D / VEC), j = (x % (D / VEC)) * VEC;
      u32x4 r = pq[u];
      if constexpr (ACT) r = act_chunk<T>(r, act_row_inv_norm<T, D / VEC>(r));
      *reinterpret_cast<u32x4*>(sQ + t * LDD + j) = r;
    }
    if constexpr (ACT) {
      // this wave's part of |SiLU(k)|^2 for every token of the sub-chunk
      for (int bb = 0; bb < NB; ++bb) {
        const f32x4 kf = silu4(Qd::f32(pk[bb]));
        float p = kf[0] * kf[0] + kf[1] * kf[1] + kf[2] * kf[2] + kf[3] * kf[3];
        p += __shfl_xor(p, 16);
        p += __shfl_xor(p, 32);
        if (g == 0) sKn[w * LW + 16 * bb + c] = p;
      }
    }
    if (tid < LW) {
      sBeta[tid] = (float)pbeta;
      if constexpr (SW) sBeta[LW + tid] = sigmoid_f((float)pws);
    }
    if (tile + 1 < ntiles) CARVE_REC_PREFETCH_Q(tile + 1);
    __syncthreads();

    // ---- P1: fold F^T[j][r] = sum_v S_hat[v][j] U[r][v] (key tile w) -----------
    if (m == 0) {
      for (int rt = 0; rt < NRT; ++rt) {
        f32x4 acc = zero4();
        for (int vp = 0; vp < D / 32; ++vp) {
          const quad a0 = Qd::ld_tr(sS, LDD, 32 * vp, 16 * w, g, c);
          const quad a1 = Qd::ld_tr(sS, LDD, 32 * vp + 16, 16 * w, g, c);
          const T* ur = sU + (16 * rt + c) * LDD + 32 * vp + 4 * g;
          acc = Qd::mma32(a0, a1, Qd::ld(ur), Qd::ld(ur + 16), acc);
        }
        Qd::st(sF + (16 * rt + c) * LDD + 16 * w + 4 * g, Qd::cvt(acc));
        Qd::st(reinterpret_cast<T*>(rec + cr.F) + (16 * rt + c) * D + 16 * w + 4 * g, Qd::cvt(acc));
      }
      __syncthreads();
    }

    // ---- P2: tau^T[r][t] = tanh(F[r] . q_t) -> sTau[t][r] -----------------------
    for (int x = w; x < NRT * NB; x += NW) {
      const int rt = x % NRT, bb = x / NRT;
      f32x4 acc = zero4();
      for (int jp = 0; jp < D / 32; ++jp) {
        const T* fr = sF + (16 * rt + c) * LDD + 32 * jp + 4 * g;
        const T* qr = sQ + (16 * bb + c) * LDD + 32 * jp + 4 * g;
        acc = Qd::mma32(Qd::ld(fr), Qd::ld(fr + 16), Qd::ld(qr), Qd::ld(qr + 16), acc);
      }
      for (int i = 0; i < 4; ++i) acc[i] = tanh_f(acc[i]);
      Qd::st(sTau + (16 * bb + c) * LDR + 16 * rt + 4 * g, Qd::cvt(acc));
      Qd::st(reinterpret_cast<T*>(rec + cr.Tau) + (m * LW + 16 * bb + c) * R2 + 16 * rt + 4 * g, Qd::cvt(acc));
    }
    __syncthreads();

    // ---- P3: gates --------------------------------------------------------------
    // key side, key tile w: lane (g, c) of block bb holds t = 16 bb + c and
    // j = 16 w + 4 g + i (i = 0..3); the prefix sums run along the 16 lanes of a row
    for (int bb = 0; bb < NB; ++bb) {
      f32x4 z = zero4();
      for (int ks = 0; ks < RP / 16; ++ks)
        z = Qd::mma16(fVb[ks], Qd::ld(sTau + (16 * bb + c) * LDR + 16 * ks + 4 * g), z);
      const f32x4 bxv = Qd::f32(pbx[bb]);
      f32x4 kv = Qd::f32(pk[bb]);
      if constexpr (ACT) {
        float n2 = 0.0f;
        for (int ww = 0; ww < NW; ++ww) n2 += sKn[ww * LW + 16 * bb + c];
        // rounded to the token dtype like the staged keys of the other kernels
        kv = Qd::f32(Qd::cvt(silu4(kv) * rsqrtf(n2 + kL2Eps)));
      }
      f32x4 gv;
      if constexpr (GATED) {
        const f32x4 fv = Qd::f32(pf[bb]);
        const f32x4 na = *reinterpret_cast<const f32x4*>(sGate + 16 * w + 4 * g);
        const f32x4 tf = *reinterpret_cast<const f32x4*>(sGate + D + 16 * w + 4 * g);
        for (int i = 0; i < 4; ++i) gv[i] = na[i] * softplus_f(fv[i] + tf[i]);
      } else {
        gv = pg[bb];
      }
      const f32x4 qv = Qd::f32(Qd::ld(sQ + (16 * bb + c) * LDD + 16 * w + 4 * g));
      f32x4 kt, qt, ki, erho, ev, sgv;
      for (int i = 0; i < 4; ++i) {
        float sp, sg;
        softplus_sigmoid(z[i] + bxv[i], sp, sg);
        const float ell = gv[i] - sp;
        const float lam = row_scan(ell);
        const float rho = 0.5f * row_bcast15(lam);
        const float E = fast_exp(lam - rho);
        // the adjoint forms Ei from the recorded E the same way (GATED: it
        // recomputes both from the gates)
        const float Ei = GATED ? fast_exp(rho - lam) : fast_rcp(E);
        // e^{lam_{-1} - rho} = e^{-rho} = Ei of the last token
        kt[i] = kv[i] * row_shr1(E, row_bcast15(Ei));
        qt[i] = qv[i] * E;
        ki[i] = kv[i] * Ei;
        erho[i] = row_bcast15(E);   // e^{lam_15 - rho} = e^{rho}
        ev[i] = E;
        sgv[i] = sg;
      }
      const int ro = (16 * bb + c) * LDD + 16 * w + 4 * g;
      Qd::st(sKt + ro, Qd::cvt(kt));
      Qd::st(sQt + ro, Qd::cvt(qt));
      Qd::st(sKi + ro, Qd::cvt(ki));
      if constexpr (!GATED) {
        // E and the erase gate of the block's tokens for the adjoint: rows of D
        const size_t re = ((size_t)(m * NB + bb) * 16 + c) * D + 16 * w + 4 * g;
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(rec + cr.E) + re) = ev;
        Qd::st(reinterpret_cast<T*>(rec + cr.Sig) + re, Qd::cvt(sgv));
      }
      if (c == 15) *reinterpret_cast<f32x4*>(sGam + bb * D + 16 * w + 4 * g) = erho;
    }
    // value side, value tile w: rows t = 16 bb + 4 g + i, column v = 16 w + c
    f32x4 wv[NB];
    for (int bb = 0; bb < NB; ++bb) {
      const f32x4 vv = Qd::mma16(ACT ? Qd::cvt(silu4(Qd::f32(pv[bb]))) : pv[bb], fI, zero4());
      if constexpr (SW) {
        const f32x4 ws = *reinterpret_cast<const f32x4*>(sBeta + LW + 16 * bb + 4 * g);
        for (int i = 0; i < 4; ++i) wv[bb][i] = ws[i] * vv[i];
      } else {
        f32x4 z = zero4();
        for (int ks = 0; ks < RP / 16; ++ks)
          z = Qd::mma16(Qd::ld(sTau + (16 * bb + c) * LDR + RP + 16 * ks + 4 * g), fVw[ks], z);
        z = Qd::mma16(pwx[bb], fI, z);                 // + wx, moved into this layout
        for (int i = 0; i < 4; ++i) wv[bb][i] = sigmoid_f(z[i]) * vv[i];
      }
    }
    if (tile + 1 < ntiles) CARVE_REC_PREFETCH_GATES(tile + 1);
    __syncthreads();

    // ---- P4: A^T and P of every block -------------------------------------------
    for (int x = w; x < 2 * NB; x += NW) {
      const bool isP = x >= NB;
      const int bb = isP ? x - NB : x;
      const T* ar = (isP ? sKi : sKt) + (16 * bb + c) * LDD + 4 * g;
      const T* br = (isP ? sQt : sKi) + (16 * bb + c) * LDD + 4 * g;
      f32x4 acc = zero4();
      for (int jp = 0; jp < D / 32; ++jp)
        acc = Qd::mma32(Qd::ld(ar + 32 * jp), Qd::ld(ar + 32 * jp + 16), Qd::ld(br + 32 * jp),
                        Qd::ld(br + 32 * jp + 16), acc);
      if (!isP) {
        // acc[i] = Kt_{t=4g+i} . Ki_{s=c}
        const f32x4 bt = *reinterpret_cast<const f32x4*>(sBeta + 16 * bb + 4 * g);
        f32x4 av;
        for (int i = 0; i < 4; ++i) av[i] = (c < 4 * g + i) ? bt[i] * acc[i] : 0.0f;
        *reinterpret_cast<f32x4*>(sAT + (bb * 16 + c) * 20 + 4 * g) = av;
      } else {
        // acc[i] = Ki_{s=4g+i} . Qt_{t=c}
        f32x4 pv4;
        for (int i = 0; i < 4; ++i) pv4[i] = (4 * g + i <= c) ? acc[i] : 0.0f;
        Qd::st(reinterpret_cast<T*>(rec + cr.P) + ((m * NB + bb) * 16 + c) * 16 + 4 * g, Qd::cvt(pv4));
      }
    }
    __syncthreads();

    // ---- P5: T = (I + A)^{-1} per block; first block's state products ------------
    // sb: S' = S diag(e^{rho}) of the block in the token dtype, the prediction's
    // operand and the record's block start state
    quad sb[NJT];
    for (int jt = 0; jt < NJT; ++jt) sb[jt] = Qd::cvt(St[jt] * *reinterpret_cast<const f32x4*>(sGam + 16 * jt + 4 * g));
    f32x4 XK = zero4();
#define CARVE_REC_XK(BB_)                                                                \
  do {                                                                                   \
    XK = zero4();                                                                        \
    const T* kr_ = sKt + (16 * (BB_) + c) * LDD + 4 * g;                                 \
    for (int jp_ = 0; jp_ < NJT / 2; ++jp_)                                              \
      XK = Qd::mma32(Qd::ld(kr_ + 32 * jp_), Qd::ld(kr_ + 32 * jp_ + 16), sb[2 * jp_],   \
                     sb[2 * jp_ + 1], XK);                                               \
  } while (0)
    if (w == NW - 1) {
      // lane (g, c): block g, row c of T, by substitution on
      //   T[c][s] = delta(c, s) - sum_{t > s} T[c][t] A[t][s],  s = 15 .. 0
      if (g < NB) {
        const float* Ab = sAT + g * 16 * 20;
        float x[16];
#pragma unroll
        for (int s = 15; s >= 0; --s) {
          float acc0 = (s == c) ? 1.0f : 0.0f, acc1 = 0.0f;
#pragma unroll
          for (int t = s + 1; t < 16; ++t) {
            if ((t - s) & 1) acc0 -= x[t] * Ab[s * 20 + t];
            else acc1 -= x[t] * Ab[s * 20 + t];
          }
          x[s] = acc0 + acc1;
        }
        T* tr = sTm + (g * 16 + c) * LDB;
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
          f32x4 t4 = {x[4 * s4], x[4 * s4 + 1], x[4 * s4 + 2], x[4 * s4 + 3]};
          Qd::st(tr + 4 * s4, Qd::cvt(t4));
          Qd::st(reinterpret_cast<T*>(rec + cr.Tm) + ((m * NB + g) * 16 + c) * 16 + 4 * s4, Qd::cvt(t4));
        }
      }
    }
    CARVE_REC_XK(0);
    __syncthreads();

    // ---- P6: token-serial blocks on the value tile (no barriers) ------------------
    for (int bb = 0; bb < NB; ++bb) {
      if (bb > 0) CARVE_REC_XK(bb);
      {
        // coalesced: quad jt of every thread is contiguous over the threads
        T* sv = reinterpret_cast<T*>(rec + cr.S) + (size_t)(m * NB + bb) * NJT * NT * 4 + tid * 4;
        for (int jt = 0; jt < NJT; ++jt) Qd::st(sv + (size_t)jt * NT * 4, sb[jt]);
      }
      const f32x4 bt = *reinterpret_cast<const f32x4*>(sBeta + 16 * bb + 4 * g);
      f32x4 rr;
      for (int i = 0; i < 4; ++i) rr[i] = bt[i] * (wv[bb][i] - XK[i]);
      const f32x4 u = Qd::mma16(Qd::ld(sTm + (bb * 16 + c) * LDB + 4 * g), Qd::cvt(rr), zero4());
      const quad uq = Qd::cvt(u);
      for (int jt = 0; jt < NJT; ++jt) {
        // S <- (S' + u^T Ki) diag(e^{rho})
        const f32x4 er = *reinterpret_cast<const f32x4*>(sGam + bb * D + 16 * jt + 4 * g);
        const f32x4 acc = Qd::mma16(Qd::ld_tr(sKi, LDD, 16 * bb, 16 * jt, g, c), uq, St[jt] * er);
        for (int i = 0; i < 4; ++i) St[jt][i] = acc[i] * er[i];
        if (bb + 1 < NB) sb[jt] = Qd::cvt(St[jt] * *reinterpret_cast<const f32x4*>(sGam + (bb + 1) * D + 16 * jt + 4 * g));
      }
    }
#undef CARVE_REC_XK
    __syncthreads();  // the next sub-chunk (or chunk) overwrites sQ, sBeta and region X
  }
#undef CARVE_REC_PREFETCH_Q
#undef CARVE_REC_PREFETCH_GATES
}

}  // namespace carve
