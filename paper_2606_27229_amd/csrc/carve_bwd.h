// carve_bwd.h -- chunked CARVE backward on gfx950 (App. Alg. backward): the
// chunk recompute + adjoint kernel templates (instantiated per variant in
// carve_variant.hip; the other launches are in carve_bwd.hip).
//
// The backward runs as a sequence of launches on one stream:
//   1. carve_sync_clear_kernel: zeroes the chunk ready flags and the ticket
//      counter of step 2 (a fill kernel, so the sequence may be graph-captured);
//   2. carve_bwd_fused_kernel: two kinds of workgroup in one grid.
//      Recompute workgroups (rec_chunk, carve_rec.h) recompute chunks
//      independently from S_chunks, latest chunks first, and write a chunk
//      record each (F, tau, T and P of every 16-token block, the block
//      retentions and the block start states), then raise that chunk's ready
//      flag.  Adjoint workgroups (bwd_adjoint below), one per (batch, head),
//      walk the chunks and their 16-token blocks in reverse, carry the state
//      gradient and wait for a chunk's flag before reading its record, so the
//      recompute runs on the compute units the adjoint leaves idle, ahead of it;
//   3. carve_bwd_param_kernel: d[Ub; Uw] from the per-chunk dF (parked in the
//      chunk records by step 2) and the chunk start states, split over
//      chunks, and dVb, dVw from dbx, dwx and tau, split over tokens;
//   4. carve_param_reduce_kernel: fixed-order sums of the parameter partials,
//      so reruns are bitwise identical.
//
// Adjoint of one 16-token block (wave w owns value tile w and key tile w; the
// state gradient dS lives in registers as dS^T tiles, rows = key index j,
// columns = the wave's 16 value rows).  The block is evaluated relative to the
// per-key-channel reference rho = lam_15 / 2, the middle of its log-retention
// range: with Sr = S diag(e^{rho}) the block start state as the chunk record
// holds it, gam = e^{lam_15 - rho} (= e^{rho}), dS' the gradient of the block
// end state (Sr + u^T Ki) diag(gam), and lam, Kt, Qt, Ki (relative to rho), A,
// P, T, R, u as in the recompute:
//   dM   = dS' diag(gam)
//   du   = Ki dM^T + P^T dO             (du_s = dM Ki_s + sum_t P_ts dO_t)
//   dR   = T^T du,  dX = -beta dR,  d(w v) = beta dR
//   dS   = (dM + dO^T Qt + dX^T Kt) diag(e^{rho})   (state gradient at the block start)
//   dKt  = dX Sr + beta dA Ki            dA = -dR u^T (s < t)
//   dQt  = dO Sr + dP Ki                 dP = dO u^T  (s <= t)
//   dKi  = diag(gam) dS'^T u + (beta dA)^T Kt + dP^T Qt
//   dbeta = rowsum(dR (w v - S Kt)) + rowsum(dA A0)    (A0 = Kt Ki^T)
//   dgam gam = gam (diag(dS'^T Sr) + sum_s Ki_s (dS'^T u_s))
//   dlam_t = dQt_t Qt_t - dKi_t Ki_t + dKt_{t+1} Kt_{t+1} + [t = 15] dgam gam
//   dl = suffix sums of dlam;  dg = dl;  dz_b = -dl b
//   dk = dKt e^{lam_{t-1} - rho} + dKi e^{rho - lam_t},  dq = dQt e^{lam_t - rho} + dY F
// rho is a constant of the block (the block's result does not depend on it), so
// the gradients through lam are those above with rho held fixed.  No factor
// exceeds e^{|lam_15| / 2}.  This kernel takes rho from its own prefix sums; the
// recompute scaled the record's Sr by its own, equal up to the rounding of the
// two evaluations of the same sums (a relative difference of order 1e-6 in the
// factors, far below the token dtype's rounding).
//   dv = d(wv) w,  dz_w = d(wv) v w (1 - w)
//   dtau = [dz_b Vb, dz_w Vw],  dY = dtau (1 - tau^2),  dF += dY^T q
// and at the chunk start the folded read-out closes the chain ("glue"):
//   dS += [Ub; Uw]^T dF,   d[Ub; Uw] += dF S_hat^T.
// With the scalar write gate (kVarScalarW; w_t = sigmoid(wx_t) on every value
// channel, no write-side content) the fold is Ub S_hat alone, there is no
// dtau_w, and the gradient of the token's write logit is the sum over the
// value channels: dwx_t = sum_v d(wv)_tv v_tv w_t (1 - w_t).
// With the input activations (kVarAct) the token tiles of q, k, v are staged
// raw; the inverse L2 norms of the block's SiLU(k), SiLU(q) rows are summed
// while staging, the quads are activated when read, and dv is taken through
// SiLU' here.  dq and dk leave this kernel as gradients of the activated q, k;
// carve_act_bwd_kernel takes them through the L2 normalisation and SiLU.
#pragma once
#include "carve_rec.h"

namespace carve {

// Bound of the ready-flag wait: 2^20 polls (each a few device-scope
// loads and a short sleep; about a second in all).  A chunk is recomputed in
// tens of microseconds by a workgroup that never waits, so the bound is not
// reached in a correct launch; if it is, the waiting wave poisons its state
// gradient with NaN (every gradient of earlier tokens then comes out NaN),
// sets the wait-timeout word of the synchronisation area and waits no more.
// The bound is a kernel argument (BwdArgs::wait_limit, kReadySpinLimit unless
// a test sets it) so that tests can make the wait give up from the host while
// every kernel still runs to completion.
// chunks whose flags one wait inspects (need, need - 1, ...)
constexpr int kReadyWindow = 8;
// how many chunks ahead of the adjoint the recompute works, and the bound of
// its wait for the adjoint's position (2^16 polls of a few hundred cycles:
// milliseconds, far beyond a chunk's time)
constexpr int kRecomputeLead = 4;
constexpr int kLeadSpinLimit = 1 << 16;

// Wait until chunk `need`'s flag is raised (flags are raised with release
// stores at agent scope) and return the lowest chunk lo such that the flags of
// chunks lo .. need, within a window of kReadyWindow chunks, were all seen
// raised; one acquire fence then covers all of them, so a wave pays for one
// cache invalidation per window instead of one per chunk.  Every lane reads
// every flag itself.  Returns need + 1 if the bound (`limit` polls) ran out.
__device__ __forceinline__ int acquire_ready(const int* rdy, const int need, const int limit) {
  for (int n = 0; n < limit; ++n) {
    // unconditional loads from clamped indices (issued back to back), masked after
    int f[kReadyWindow];
#pragma unroll
    for (int i = 0; i < kReadyWindow; ++i)
      f[i] = __hip_atomic_load(rdy + (need - i >= 0 ? need - i : 0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int i = 1; i < kReadyWindow; ++i)
      if (need - i < 0) f[i] = 0;
    if (f[0] != 0) {
      int lo = need;
#pragma unroll
      for (int i = 1; i < kReadyWindow; ++i) {
        if (f[i] == 0) break;
        lo = need - i;
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      return lo;
    }
    __builtin_amdgcn_s_sleep(2);
  }
  return need + 1;
}

// Compiler-only fence: keeps the LDS loads of one loop iteration from being
// hoisted above the previous one (bounds the number of live operand registers).
#define CARVE_SEQ() asm volatile("" ::: "memory")

// Adjoint of (batch, head) bh.  ready[bh * nch + ch] is raised when chunk ch's
// record is complete; smem is the workgroup's dynamic LDS (BwdLds layout).
// GATED: g is formed from its staged raw logit f (Eq. decay_gate); the kernel
// writes df = dg (-exp(A)) sigmoid(f + tau_f) instead of dg and sums dA = dg g
// and dtau = df over its tokens (per lane in registers, reduced once at the
// end) into a per-(batch, head) partial.
template <typename T, int D, int RP, int VAR>
__device__ __forceinline__ void bwd_adjoint(const BwdArgs& a, const int bh, char* smem, const int* ready,
                                            int* timeout_word, int* pos) {
  typedef Quad<T> Qd;
  typedef typename Qd::q quad;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr bool GATED = (VAR & kVarGated) != 0;
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr bool ACT = (VAR & kVarAct) != 0;
  constexpr int NT = bwd_threads(D);
  constexpr int NW = NT / 64;
  constexpr int NJT = D / 16;
  constexpr int R2 = fold_rows(RP, VAR);
  constexpr int NRT = R2 / 16;
  constexpr int NRB = RP / 16;
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDD = D + PAD, LDR = R2 + PAD, LDB = 16 + PAD;
  // bank-conflict-free layouts (QS): Kt, Qt, Ki, VbT, VwT rows of LDK and the
  // exchange tiles rows of LDX with the quad swizzle (qx), S and dS' rows of
  // LDSX (SXH, bf16 d = 128: unpadded with hswz128)
  constexpr bool QS = bwd_qswz<T, VAR>(), SXH = bwd_sx_hswz<T, D, VAR>();
  constexpr int LDK = bwd_ldk<T, D, VAR>(), LDX = bwd_ldx<T, VAR>(), LDSX = bwd_ldsx<T, D, VAR>();
  constexpr int VEC = 16 / sizeof(T);
  static_assert(NW == NJT, "one wave per 16-wide tile");

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  // the quad-swizzle term of row r, and the transposing operand read, of the
  // tiles laid out with QS
#define CARVE_QX(R_) (QS ? qswz<T>(R_) : 0)
#define CARVE_LDTR(B_, LD_, R0_, C0_) (QS ? Qd::ld_tr_sw(B_, LD_, R0_, C0_, g, c) : Qd::ld_tr(B_, LD_, R0_, C0_, g, c))
  const int H = a.H, Tn = a.T, L = a.L, R = a.R;
  const int b = bh / H, h = bh % H;
  const int nch = Tn / L, nbc = L / 16;

  constexpr BwdLds lay = bwd_lds<T, D, RP, VAR>();
  constexpr int NS = bwd_stage_tiles(SW);             // staged token tiles per block
  // the key-side factors of a block (E and the erase gate) come from the
  // chunk record, staged in place of g and bx; GATED kernels recompute them
  // from f, bx and tau
  constexpr bool KREC = !GATED;
  T* sF = reinterpret_cast<T*>(smem + lay.F);        // [R2][LDD]    F of the chunk
  T* sVbT = reinterpret_cast<T*>(smem + lay.VbT);    // [RP][LDK]    Vb^T (quad-swizzled)
  T* sVwT = reinterpret_cast<T*>(smem + lay.VwT);    // [RP][LDK]    Vw^T (not SW; quad-swizzled)
  T* sTau = reinterpret_cast<T*>(smem + lay.Tau);    // [16][LDR]    tau of the block
  T* sTm = reinterpret_cast<T*>(smem + lay.Tm);      // [16][LDB]    T of the block
  T* sP = reinterpret_cast<T*>(smem + lay.P);        // [16][LDB]    P of the block
  float* sGam = reinterpret_cast<float*>(smem + lay.Gam);      // [D] gam = e^{rho} of the block
  float* sBeta = reinterpret_cast<float*>(smem + lay.Beta);    // [16] beta, then [16] sigmoid(wx) (SW)
  float* sDbeta = reinterpret_cast<float*>(smem + lay.Dbeta);  // [NW + 1][16]
  float* sDwx = reinterpret_cast<float*>(smem + lay.Dwx);      // [NW][16] (SW)
  float* sInv = reinterpret_cast<float*>(smem + lay.Inv);      // [2][16] 1/|SiLU(k)|, 1/|SiLU(q)| (ACT)
  T* sKt = reinterpret_cast<T*>(smem + lay.Kt);      // [16][LDK]    (quad-swizzled)
  T* sQt = reinterpret_cast<T*>(smem + lay.Qt);      // [16][LDK]
  T* sKi = reinterpret_cast<T*>(smem + lay.Ki);      // [16][LDK]
  T* sSx = reinterpret_cast<T*>(smem + lay.Sx);      // [D][LDSX]    S[v][j] (block start)
  T* sdSx = reinterpret_cast<T*>(smem + lay.dSx);    // [D][LDSX]    dS'[v][j]; glue: dF at (j, r)
  T* sdOT = reinterpret_cast<T*>(smem + lay.dOT);    // [D][LDX]     [value][token] exchange (quad-swizzled)
  T* suT = reinterpret_cast<T*>(smem + lay.uT);
  T* sdRT = reinterpret_cast<T*>(smem + lay.dRT);
  T* sdzwT = reinterpret_cast<T*>(smem + lay.dzwT);
  T* sdzb = reinterpret_cast<T*>(smem + lay.dzb);    // [16][LDD]    dz_b[t][j]
  T* sdY = reinterpret_cast<T*>(smem + lay.dY);      // [16][LDR]    dY[t][r]
  T* sStg = reinterpret_cast<T*>(smem + lay.Stage);  // [NS][16][D]  token tiles, swizzled
  float* sGs = reinterpret_cast<float*>(smem + lay.Stage + lds_round(NS * 16 * D * sizeof(T)));  // [16][D] g

  const size_t bh0 = ((size_t)b * Tn * H + h) * D;
  const size_t bh1 = (size_t)b * Tn * H + h;
  const int rs = H * D;
  const T* __restrict__ q = reinterpret_cast<const T*>(a.q) + bh0;
  const T* __restrict__ k = reinterpret_cast<const T*>(a.k) + bh0;
  const T* __restrict__ v = reinterpret_cast<const T*>(a.v) + bh0;
  const T* __restrict__ bx = reinterpret_cast<const T*>(a.bx) + bh0;
  const T* __restrict__ wx = reinterpret_cast<const T*>(a.wx) + (SW ? bh1 : bh0);
  const T* __restrict__ beta = reinterpret_cast<const T*>(a.beta) + bh1;
  const T* __restrict__ dO = reinterpret_cast<const T*>(a.dO) + bh0;
  const float* __restrict__ gl = GATED ? nullptr : a.g + bh0;
  const T* __restrict__ fl = GATED ? reinterpret_cast<const T*>(a.f) + bh0 : nullptr;
  T* __restrict__ dq = reinterpret_cast<T*>(a.dq) + bh0;
  T* __restrict__ dk = reinterpret_cast<T*>(a.dk) + bh0;
  T* __restrict__ dv = reinterpret_cast<T*>(a.dv) + bh0;
  T* __restrict__ dbx = reinterpret_cast<T*>(a.dbx) + bh0;
  T* __restrict__ dwx = reinterpret_cast<T*>(a.dwx) + (SW ? bh1 : bh0);
  T* __restrict__ dbeta = reinterpret_cast<T*>(a.dbeta) + bh1;
  float* __restrict__ dgo = GATED ? nullptr : a.dg + bh0;
  T* __restrict__ dfo = GATED ? reinterpret_cast<T*>(a.df) + bh0 : nullptr;
  float* sGate = reinterpret_cast<float*>(smem + lay.Gate);   // [2][D] -exp(A), tau_f (GATED)
  T* sFs = reinterpret_cast<T*>(sGs);                          // [16][D] staged f (GATED)
  const ChunkRec cr = chunk_rec(sizeof(T), D, L, R2);
  const char* recb = reinterpret_cast<const char*>(a.rec) + (size_t)bh * nch * cr.total;

  // ---- shared parameters ------------------------------------------------------
  for (int x = tid; x < RP * D; x += NT) {
    const int rr = x / D, j = x % D;
    sVbT[rr * LDK + (j ^ CARVE_QX(rr))] = (T)(rr < R ? a.Vb[j * R + rr] : 0.0f);
    if constexpr (!SW) sVwT[rr * LDK + (j ^ CARVE_QX(rr))] = (T)(rr < R ? a.Vw[j * R + rr] : 0.0f);
  }
  // Vb / Vw operand quads (lane (g, c): V[16 w + c][16 ks + 4 g + e]) are read
  // from sVbT / sVwT with the transposing load where needed; the identity
  // operand (lane (g, c): I[4 g + e][c]) is rebuilt where needed.
  if (GATED)
    for (int x = tid; x < D; x += NT) {
      sGate[x] = -expf(a.A[h * D + x]);
      sGate[D + x] = a.tau_f[h * D + x];
    }
#define CARVE_FVB(KS_) CARVE_LDTR(sVbT, LDK, 16 * (KS_), 16 * w)
#define CARVE_FVW(KS_) CARVE_LDTR(sVwT, LDK, 16 * (KS_), 16 * w)
#define CARVE_FI() Qd::cvt(f32x4{4 * g == c ? 1.0f : 0.0f, 4 * g + 1 == c ? 1.0f : 0.0f, \
                                 4 * g + 2 == c ? 1.0f : 0.0f, 4 * g + 3 == c ? 1.0f : 0.0f})
  __syncthreads();

  // ---- persistent accumulators --------------------------------------------------
  const size_t soff = (size_t)bh * D * D;
  f32x4 dSt[NJT];                 // dS[v = 16 w + c][j = 16 jt + 4 g + i]
  for (int jt = 0; jt < NJT; ++jt)
    dSt[jt] = a.dS_T ? gload4(a.dS_T + soff + (16 * w + c) * D + 16 * jt + 4 * g) : zero4();
  f32x4 dF[NRT];                  // dF[r = 16 rt + 4 g + i][j = 16 w + c]
  // GATED: this lane's sums over its tokens of dg g and df (channels 16 w + 4 g + i)
  f32x4 gaccA = zero4(), gaccT = zero4();
  for (int rt = 0; rt < NRT; ++rt) dF[rt] = zero4();

  // ---- prefetch registers: the next block to process (reverse order) and, at
  // the last block of a chunk, the fold F of the next chunk.  Every block
  // starts with one wait for all of this wave's memory operations, issued at
  // least a block earlier.
  constexpr int NTAU = 16 * R2 / VEC;   // 16-byte vectors of a block's tau
  constexpr int NTV = (NTAU + NT - 1) / NT;
  constexpr int NFV = (R2 * D / VEC + NT - 1) / NT;   // 16-byte vectors of F per thread
  u32x4 ptau[NTV], pF[NFV];
  // token tiles k, q, bx (KREC: the recorded erase gate), v, dO and (not SW) wx
  // of a block: NS * 16 rows of D elements read as 16-byte vectors (whole rows,
  // coalesced) and staged through LDS
  constexpr int NC = D / VEC;                    // 16-byte chunks per row
  constexpr int NSV = NS * 16 * NC;              // vectors of the tiles
  constexpr int NSTG = (NSV + NT - 1) / NT;      // per thread
  static_assert((16 * NC) % 64 == 0 || NSV % NT == 0, "tile index uniform per wave");
  static_assert(!ACT || (16 * NC) % 64 == 0, "a staged row's chunks in one wave (row sums over lanes)");
  u32x4 pstg[NSTG];
  // g (KREC: the recorded E) of a block: 16 rows of D floats, one 16-byte
  // vector per thread
  constexpr int NGC = D / 4;                     // 16-byte chunks per g row
  static_assert(16 * NGC == NT, "one g vector per thread");
  quad ptm, ppm, psbq[NJT];
  f32x4 pg;
  u32x4 pfv;        // a 16-byte vector of the block's f rows (GATED)
  T pbeta = (T)0.0f, pws = (T)0.0f;   // beta and (SW) the write logit of token tid
  // The prefetch of a block is issued in two parts during the previous block's
  // value- and key-side steps (which hardly use the memory pipeline), not at
  // its top, where issuing it would stall the waves: LOADA (token tiles, tau,
  // T, P, retention, beta, g) and LOADS (the block start state, once the
  // current one has had its last use).
#define CARVE_BWD_LOADS(GB_)                                                                  \
  do {                                                                                        \
    const int ch_ = (GB_) / nbc, bc_ = (GB_) % nbc;                                           \
    const char* rc_ = recb + (size_t)ch_ * cr.total;                                          \
    const T* sv_ = reinterpret_cast<const T*>(rc_ + cr.S) + (size_t)bc_ * NJT * NT * 4 + tid * 4; \
    for (int jt_ = 0; jt_ < NJT; ++jt_) psbq[jt_] = Qd::ld(sv_ + (size_t)jt_ * NT * 4);        \
  } while (0)
#define CARVE_BWD_LOADA(GB_)                                                                  \
  do {                                                                                        \
    const int ch_ = (GB_) / nbc, bc_ = (GB_) % nbc;                                           \
    const char* rc_ = recb + (size_t)ch_ * cr.total;                                          \
    const int tb_ = ch_ * L + 16 * bc_;                                                       \
    const int e_ = (tb_ + c) * rs + 16 * w + 4 * g;                                           \
    const T* tau_ = reinterpret_cast<const T*>(rc_ + cr.Tau) + 16 * bc_ * R2;                 \
    for (int u_ = 0; u_ < NTV; ++u_) {                                                        \
      const int x_ = tid + u_ * NT;                                                           \
      if (x_ < NTAU) ptau[u_] = *reinterpret_cast<const u32x4*>(tau_ + x_ * VEC);             \
    }                                                                                         \
    if (tid < 64) {                                                                           \
      ptm = Qd::ld(reinterpret_cast<const T*>(rc_ + cr.Tm) + bc_ * 256 + 4 * tid);            \
      ppm = Qd::ld(reinterpret_cast<const T*>(rc_ + cr.P) + bc_ * 256 + 4 * tid);             \
    }                                                                                         \
    if (tid < 16) {                                                                           \
      pbeta = beta[(tb_ + tid) * H];                                                          \
      if constexpr (SW) pws = wx[(tb_ + tid) * H];                                            \
    }                                                                                         \
    for (int u_ = 0; u_ < NSTG; ++u_) {                                                       \
      const int x_ = tid + u_ * NT;                                                           \
      if (NSV % NT != 0 && x_ >= NSV) break;                                                  \
      const int s_ = x_ / (16 * NC), t_ = (x_ / NC) % 16, k_ = x_ % NC;                       \
      if (KREC && s_ == 2) {                                                                  \
        /* the recorded erase gate of the block (rows of D) in place of bx */                 \
        pstg[u_] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(rc_ + cr.Sig) +   \
                                                   (16 * bc_ + t_) * D + k_ * VEC);            \
      } else {                                                                                \
        const T* src_ = s_ == 0 ? k : s_ == 1 ? q : s_ == 2 ? bx : s_ == 3 ? v : s_ == 4 ? dO : wx; \
        pstg[u_] = *reinterpret_cast<const u32x4*>(src_ + (tb_ + t_) * rs + k_ * VEC);         \
      }                                                                                       \
    }                                                                                         \
    if constexpr (GATED) {                                                                    \
      if (tid < 16 * NC) pfv = *reinterpret_cast<const u32x4*>(fl + (tb_ + tid / NC) * rs + (tid % NC) * VEC); \
    } else {                                                                                  \
      /* the recorded E of the block in place of g */                                          \
      pg = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(rc_ + cr.E) +         \
                                           (16 * bc_ + tid / NGC) * D + 4 * (tid % NGC));      \
    }                                                                                         \
    (void)e_;                                                                                 \
  } while (0)
#define CARVE_BWD_LOADF(CH_)                                                                  \
  do {                                                                                        \
    const T* src_ = reinterpret_cast<const T*>(recb + (size_t)(CH_) * cr.total + cr.F);       \
    for (int u_ = 0; u_ < NFV; ++u_) {                                                        \
      const int x_ = tid + u_ * NT;                                                           \
      if (x_ < R2 * D / VEC) pF[u_] = *reinterpret_cast<const u32x4*>(src_ + x_ * VEC);       \
    }                                                                                         \
  } while (0)
  // [Ub; Uw] operand quads of the glue, lane (g, c): U[16 rt + 4 g + e][16 w + c]
  // (rows past R are zero), loaded once for the whole call
  quad fU[NRT];
  for (int rt = 0; rt < NRT; ++rt) {
    const float* src = rt < RP / 16 ? a.Ub : a.Uw;
    f32x4 tu;
    for (int e = 0; e < 4; ++e) {
      const int rl = 16 * (rt % (RP / 16)) + 4 * g + e;
      tu[e] = rl < R ? src[rl * D + 16 * w + c] : 0.0f;
    }
    fU[rt] = Qd::cvt(tu);
  }
  const int ngb = nch * nbc;
  const int* rdy = ready + (size_t)bh * nch;
  // chunks >= acq_lo have been acquired by this wave; acq_lo = -1 after a wait
  // ran out of its bound (never in a correct launch)
  int acq_lo = nch;
#define CARVE_BWD_READY(CH_)                                                                  \
  do {                                                                                        \
    if ((CH_) < acq_lo) {                                                                     \
      const int lo_ = acquire_ready(rdy, (CH_), a.wait_limit);                                \
      if (lo_ > (CH_)) {                                                                      \
        acq_lo = -1;                                                                          \
        if ((threadIdx.x & 63) == 0)                                                          \
          __hip_atomic_store(timeout_word, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);    \
        for (int jt_ = 0; jt_ < NJT; ++jt_) dSt[jt_] = f32x4{__builtin_nanf(""), __builtin_nanf(""), \
                                                             __builtin_nanf(""), __builtin_nanf("")}; \
      } else {                                                                                \
        acq_lo = lo_;                                                                         \
      }                                                                                       \
    }                                                                                         \
  } while (0)
  CARVE_BWD_READY(nch - 1);
  CARVE_BWD_LOADA(ngb - 1);
  CARVE_BWD_LOADS(ngb - 1);
  CARVE_BWD_LOADF(nch - 1);

  // pending dq / dF update of the last processed block (its BQ step)
  f32x4 pdqp = zero4();
  quad pqq = Qd::cvt(zero4());
  int pe0 = 0;
#define CARVE_BWD_BQ()                                                                        \
  do {                                                                                        \
    f32x4 acc_ = pdqp;                                                                        \
    for (int rp = 0; rp < R2 / 32; ++rp)                                                      \
      acc_ = Qd::mma32(Qd::ld_tr(sF, LDD, 32 * rp, 16 * w, g, c), Qd::ld_tr(sF, LDD, 32 * rp + 16, 16 * w, g, c), \
                       Qd::ld(sdY + c * LDR + 32 * rp + 4 * g), Qd::ld(sdY + c * LDR + 32 * rp + 16 + 4 * g), acc_); \
    Qd::st(dq + pe0, Qd::cvt(acc_));                                                          \
    const quad qT_ = Qd::cvt(Qd::mma16(pqq, CARVE_FI(), zero4()));   /* q[t = 4g + i][j = 16 w + c] */ \
    for (int rt = 0; rt < NRT; ++rt) dF[rt] = Qd::mma16(Qd::ld_tr(sdY, LDR, 0, 16 * rt, g, c), qT_, dF[rt]); \
  } while (0)
#define CARVE_BWD_GAM()                                                                       \
  do {                                                                                        \
    f32x4 gm_[NJT];                                                                           \
    for (int jt_ = 0; jt_ < NJT; ++jt_) gm_[jt_] = *reinterpret_cast<const f32x4*>(sGam + 16 * jt_ + 4 * g); \
    for (int jt_ = 0; jt_ < NJT; ++jt_) dSt[jt_] *= gm_[jt_];                                 \
  } while (0)
#pragma unroll 1
  for (int gb = ngb - 1; gb >= 0; --gb) {
    const int ch = gb / nbc, bc = gb % nbc;
    const char* rc = recb + (size_t)ch * cr.total;
    {
      // opaque copies of the lane coordinates: values derived from them
      // (addresses, masks) are recomputed in every block instead of being
      // hoisted out of the loops and kept live (which would spill)
      int tid_ = tid, g_ = g, c_ = c, w_ = w;
      asm volatile("" : "+v"(tid_), "+v"(g_), "+v"(c_), "+v"(w_));
      const int tid = tid_, g = g_, c = c_, w = w_;
      const int lane = tid & 63;
      (void)lane;
      const int tb = ch * L + 16 * bc;   // first token of the block
      const int e0 = (tb + c) * rs + 16 * w + 4 * g;

      // -- BK1 (a): this block's data (prefetched a block ago) ------------------------
      vm_wait_all();
      u32x4 ltau[NTV];
      for (int u = 0; u < NTV; ++u) ltau[u] = ptau[u];
      const quad ltm = ptm, lpm = ppm;
      const T lbeta = pbeta, lws = pws;
      quad sbq[NJT];   // block start state, wave layout: S[16 w + c][16 jt + 4 g + e]
      for (int jt = 0; jt < NJT; ++jt) sbq[jt] = psbq[jt];
      {
        // S of the block into its own region now (the last block's key side,
        // its only reader, ended two barriers ago); dS' waits for the first
        // barrier (its region holds the glue's dF parts until then)
        const int hx = SXH ? hswz128(c) : 0;
        for (int jt = 0; jt < NJT; ++jt) Qd::st(sSx + (16 * w + c) * LDSX + ((16 * jt + 4 * g) ^ hx), sbq[jt]);
      }
      u32x4 lstg[NSTG];
      for (int u = 0; u < NSTG; ++u) lstg[u] = pstg[u];
      const f32x4 lg_row = pg;   // a row vector of g (staged below)
      const u32x4 lf_row = pfv;  // GATED: a row vector of f
      if (bc == nbc - 1) {
        // first block of a chunk in reverse order: the chunk's F into LDS (the
        // previous chunk's last read of sF was before its glue barriers)
        for (int u = 0; u < NFV; ++u) {
          const int x = tid + u * NT;
          if (x < R2 * D / VEC) {
            const int rr = x / (D / VEC), j = (x % (D / VEC)) * VEC;
            *reinterpret_cast<u32x4*>(sF + rr * LDD + j) = pF[u];
          }
        }
      }
      // the next block's prefetch (below) reads chunk ch - 1's record at a
      // chunk's last block: wait until the recompute has published it
      if (bc == 0 && ch > 0) CARVE_BWD_READY(ch - 1);

      // -- BQ of the previous block (overlaps the loads above) -------------------
      if (bc < nbc - 1) CARVE_BWD_BQ();

      // -- BK1 (c): stage the block record; recompute the key side; S, dS' -> LDS
      for (int u = 0; u < NTV; ++u) {
        const int x = tid + u * NT;
        if (x < NTAU) {
          const int t = x / (R2 / VEC), r = (x % (R2 / VEC)) * VEC;
          *reinterpret_cast<u32x4*>(sTau + t * LDR + r) = ltau[u];
        }
      }
      if (tid < 64) {
        const int t = tid >> 2, s4 = 4 * (tid & 3);
        Qd::st(sTm + t * LDB + s4, ltm);
        Qd::st(sP + t * LDB + s4, lpm);
      }
      if (tid < 16) {
        sBeta[tid] = (float)lbeta;
        if constexpr (SW) sBeta[16 + tid] = sigmoid_f((float)lws);
      }
      // token tiles -> LDS: 16-byte chunk kk of row t goes to chunk kk ^ (t mod NC)
      // (a row-dependent swizzle instead of padding: the 16 rows a wave reads in
      // one quad load fall into distinct banks)
      for (int u = 0; u < NSTG; ++u) {
        const int x = tid + u * NT;
        if (NSV % NT != 0 && x >= NSV) break;
        const int s_ = x / (16 * NC), t = (x / NC) % 16, kk = x % NC;
        *reinterpret_cast<u32x4*>(sStg + (s_ * 16 + t) * D + (kk ^ (t & (NC - 1))) * VEC) = lstg[u];
        if constexpr (ACT) {
          // k (s_ = 0) and q (s_ = 1) rows: the row's NC chunks are in NC
          // consecutive lanes, and s_ is uniform over a wave
          if (s_ < 2) {
            const float inv = act_row_inv_norm<T, NC>(lstg[u]);
            if (kk == 0) sInv[s_ * 16 + t] = inv;
          }
        }
      }
      if constexpr (GATED) {
        if (tid < 16 * NC) {
          const int t = tid / NC, kk = tid % NC;
          *reinterpret_cast<u32x4*>(sFs + t * D + (kk ^ (t & (NC - 1))) * VEC) = lf_row;
        }
      } else {
        const int t = tid / NGC, kk = tid % NGC;
        *reinterpret_cast<f32x4*>(sGs + t * D + 4 * (kk ^ (t & (NGC - 1)))) = lg_row;
      }
      // the previous block's state gradient with respect to S (the factor
      // e^{rho} of its sGam, which the form step below rewrites); deferred
      // from that block's end, where its loads would wait one by one
      if (bc < nbc - 1) CARVE_BWD_GAM();
      __syncthreads();
      // the chunks started so far, for the pacing of the recompute
      if (bc == nbc - 1 && tid == 0) __hip_atomic_store(pos, nch - ch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // this wave's quads of the token tiles (row t = c, elements 16 w + 4 g ..
      // + 3) and of tau_b; read before the barrier that ends this step, so the
      // value-side step may overwrite the staging region
      quad kq, qq, lbx, vq, wxq, dOq, ltq[NRB];
      quad vraw;  // ACT: the raw value quad (for SiLU' of dv)
      f32x4 lg;
      {
        const int by = (16 * w + 4 * g) * (int)sizeof(T);
        const int off = ((((by >> 4) ^ (c & (NC - 1))) << 4) | (by & 15)) / (int)sizeof(T);
        if constexpr (GATED) {
          const f32x4 fv = Qd::f32(Qd::ld(sFs + c * D + off));
          const f32x4 na = *reinterpret_cast<const f32x4*>(sGate + 16 * w + 4 * g);
          const f32x4 tf = *reinterpret_cast<const f32x4*>(sGate + D + 16 * w + 4 * g);
          for (int i = 0; i < 4; ++i) lg[i] = na[i] * softplus_f(fv[i] + tf[i]);
        } else {
          lg = *reinterpret_cast<const f32x4*>(sGs + c * D + 4 * ((4 * w + g) ^ (c & (NGC - 1))));
        }
        const T* r0 = sStg + c * D + off;
        kq = Qd::ld(r0);
        qq = Qd::ld(r0 + 16 * D);
        lbx = Qd::ld(r0 + 32 * D);
        vq = Qd::ld(r0 + 48 * D);
        dOq = Qd::ld(r0 + 64 * D);
        if constexpr (!SW) wxq = Qd::ld(r0 + 80 * D);
        if constexpr (ACT) {
          kq = Qd::cvt(silu4(Qd::f32(kq)) * sInv[c]);
          qq = Qd::cvt(silu4(Qd::f32(qq)) * sInv[16 + c]);
          vraw = vq;
          vq = Qd::cvt(silu4(Qd::f32(vq)));
        }
        if constexpr (!KREC)
          for (int ks = 0; ks < NRB; ++ks) ltq[ks] = Qd::ld(sTau + c * LDR + 16 * ks + 4 * g);
      }
      // key-side factors kept for the adjoint in the token dtype (quads)
      quad Eq, Eiq, sigq;
      {
        const f32x4 kv = Qd::f32(kq), qv = Qd::f32(qq);
        f32x4 kt, qt, ki, E, Ei, sig, gp;
        if constexpr (KREC) {
          // E and the erase gate as the recompute formed them (staged in place
          // of g and bx); Ei from E as there, so every tile matches its T and P
          sig = Qd::f32(lbx);
          for (int i = 0; i < 4; ++i) {
            E[i] = lg[i];
            Ei[i] = fast_rcp(E[i]);
          }
        } else {
          f32x4 z = zero4();
          for (int ks = 0; ks < NRB; ++ks) z = Qd::mma16(CARVE_FVB(ks), ltq[ks], z);
          const f32x4 bxv = Qd::f32(lbx);
          for (int i = 0; i < 4; ++i) {
            float sp, sg;
            softplus_sigmoid(z[i] + bxv[i], sp, sg);
            sig[i] = sg;
            const float lam = row_scan(lg[i] - sp);
            const float rho = 0.5f * row_bcast15(lam);
            E[i] = fast_exp(lam - rho);
            Ei[i] = fast_exp(rho - lam);
          }
        }
        for (int i = 0; i < 4; ++i) {
          // e^{lam_{-1} - rho} = e^{-rho} = Ei of the last token
          kt[i] = kv[i] * row_shr1(E[i], row_bcast15(Ei[i]));
          qt[i] = qv[i] * E[i];
          ki[i] = kv[i] * Ei[i];
          gp[i] = row_bcast15(E[i]);   // gam = e^{lam_15 - rho} = e^{rho}
        }
        if (c == 0) *reinterpret_cast<f32x4*>(sGam + 16 * w + 4 * g) = gp;
        Eq = Qd::cvt(E);
        Eiq = Qd::cvt(Ei);
        sigq = Qd::cvt(sig);
        const int ro = c * LDK + 16 * w + ((4 * g) ^ CARVE_QX(c));
        Qd::st(sKt + ro, Qd::cvt(kt));
        Qd::st(sQt + ro, Qd::cvt(qt));
        Qd::st(sKi + ro, Qd::cvt(ki));
      }
      {
        // row 16 w + c: its swizzle term depends on c only
        const int hx = SXH ? hswz128(c) : 0;
        for (int jt = 0; jt < NJT; ++jt) {
          const int o = (16 * w + c) * LDSX + ((16 * jt + 4 * g) ^ hx);
          Qd::st(sdSx + o, Qd::cvt(dSt[jt]));
        }
      }
      if constexpr (KREC) {
        // dS' becomes dM = dS' diag(gam) in place, gam = e^{rho} = E of the
        // block's last token (row 15 of the staged record: the same values
        // the form step above writes to sGam for its own key tile)
        f32x4 gm[NJT];
        for (int jt = 0; jt < NJT; ++jt)
          gm[jt] = *reinterpret_cast<const f32x4*>(sGs + 15 * D + 4 * ((4 * jt + g) ^ (15 & (NGC - 1))));
        for (int jt = 0; jt < NJT; ++jt) dSt[jt] *= gm[jt];
      }
      __syncthreads();

      // -- BV: value-side adjoint (value tile w, rows t = 4 g + i, column v = 16 w + c)
      // prefetch (part A) of the next block, and at a chunk's last block the
      // next chunk's F
      CARVE_BWD_LOADA(gb > 0 ? gb - 1 : 0);
      if (bc == 0) CARVE_BWD_LOADF(ch > 0 ? ch - 1 : 0);
      {
        const f32x4 vv = Qd::mma16(vq, CARVE_FI(), zero4());
        const f32x4 dOc = Qd::mma16(dOq, CARVE_FI(), zero4());
        f32x4 wgt;
        if constexpr (SW) {
          wgt = *reinterpret_cast<const f32x4*>(sBeta + 16 + 4 * g);   // one gate per token
        } else {
          f32x4 zw = zero4();
          for (int ks = 0; ks < NRB; ++ks)
            zw = Qd::mma16(Qd::ld(sTau + c * LDR + RP + 16 * ks + 4 * g), CARVE_FVW(ks), zw);
          zw = Qd::mma16(wxq, CARVE_FI(), zw);
          for (int i = 0; i < 4; ++i) wgt[i] = sigmoid_f(zw[i]);
        }
        f32x4 XK = zero4();
        const T* kr = sKt + c * LDK + ((4 * g) ^ CARVE_QX(c));
        for (int jp = 0; jp < NJT / 2; ++jp)
          XK = Qd::mma32(Qd::ld(kr + 32 * jp), Qd::ld(kr + 32 * jp + 16), sbq[2 * jp], sbq[2 * jp + 1], XK);
        const f32x4 bt = *reinterpret_cast<const f32x4*>(sBeta + 4 * g);
        f32x4 rm, rr;
        for (int i = 0; i < 4; ++i) {
          rm[i] = wgt[i] * vv[i] - XK[i];
          rr[i] = bt[i] * rm[i];
        }
        const f32x4 u = Qd::mma16(Qd::ld(sTm + c * LDB + 4 * g), Qd::cvt(rr), zero4());
        // du = Ki dM^T + P^T dO with dM = dS' diag(gam)
        f32x4 du = zero4();
        const T* kir = sKi + c * LDK + ((4 * g) ^ CARVE_QX(c));
        // dS' (already in LDS for the key side) becomes dM in place (KREC: in
        // the form step): both du and the state gradient below use dM only
        if constexpr (!KREC)
          for (int jt = 0; jt < NJT; ++jt) dSt[jt] *= *reinterpret_cast<const f32x4*>(sGam + 16 * jt + 4 * g);
        for (int jp = 0; jp < NJT / 2; ++jp)
          du = Qd::mma32(Qd::ld(kir + 32 * jp), Qd::ld(kir + 32 * jp + 16), Qd::cvt(dSt[2 * jp]),
                         Qd::cvt(dSt[2 * jp + 1]), du);
        const quad dOcq = Qd::cvt(dOc);
        du = Qd::mma16(Qd::ld_tr(sP, LDB, 0, 0, g, c), dOcq, du);
        const f32x4 dR = Qd::mma16(Qd::ld_tr(sTm, LDB, 0, 0, g, c), Qd::cvt(du), zero4());
        f32x4 dX, dwv;
        for (int i = 0; i < 4; ++i) {
          dX[i] = -bt[i] * dR[i];
          dwv[i] = bt[i] * dR[i];
        }
        const quad dXq = Qd::cvt(dX);
        // state gradient at the block start
        for (int jt = 0; jt < NJT; ++jt) {
          CARVE_SEQ();
          dSt[jt] = Qd::mma32(CARVE_LDTR(sQt, LDK, 0, 16 * jt), CARVE_LDTR(sKt, LDK, 0, 16 * jt), dOcq,
                              dXq, dSt[jt]);
        }
        // value-side token gradients, stored through the identity (4 values per lane)
        f32x4 dvv, dzw;
        for (int i = 0; i < 4; ++i) {
          dvv[i] = dwv[i] * wgt[i];
          dzw[i] = dwv[i] * vv[i] * wgt[i] * (1.0f - wgt[i]);
        }
        if constexpr (ACT)
          Qd::st(dv + e0, Qd::cvt(Qd::mma16(Qd::cvt(dvv), CARVE_FI(), zero4()) * silu_grad4(Qd::f32(vraw))));
        else
          Qd::st(dv + e0, Qd::cvt(Qd::mma16(Qd::cvt(dvv), CARVE_FI(), zero4())));
        const quad dzwq = Qd::cvt(dzw);
        if constexpr (SW) {
          // the token's write-logit gradient, partial over this wave's 16 values
          f32x4 pw;
          for (int i = 0; i < 4; ++i) pw[i] = row_scan(dzw[i]);
          if (c == 15) *reinterpret_cast<f32x4*>(sDwx + w * 16 + 4 * g) = pw;
        } else {
          Qd::st(dwx + e0, Qd::cvt(Qd::mma16(dzwq, CARVE_FI(), zero4())));
        }
        // beta gradient, value part: sum over v of dR (w v - S Kt)
        f32x4 pr;
        for (int i = 0; i < 4; ++i) pr[i] = row_scan(dR[i] * rm[i]);
        if (c == 15) *reinterpret_cast<f32x4*>(sDbeta + w * 16 + 4 * g) = pr;
        // exchange, [value][token] layout
        const int xo = (16 * w + c) * LDX + ((4 * g) ^ CARVE_QX(c));
        Qd::st(sdRT + xo, Qd::cvt(dR));
        Qd::st(sdOT + xo, dOcq);
        Qd::st(suT + xo, Qd::cvt(u));
        if constexpr (!SW) Qd::st(sdzwT + xo, dzwq);
      }
      __syncthreads();

      // -- BKA: key-side adjoint (key tile w; C rows j = 16 w + 4 g + i, column t = c)
      // prefetch (part S): the next block's start state (sbq had its last use in BV)
      CARVE_BWD_LOADS(gb > 0 ? gb - 1 : 0);
      f32x4 dqp;
      {
        const f32x4 E = Qd::f32(Eq), Ei = Qd::f32(Eiq), sig = Qd::f32(sigq);
        f32x4 dKt = zero4(), dQt = zero4(), dKi = zero4(), dA = zero4(), dP = zero4();
        float dgs = 0.0f;   // sum_v dS'[v][j] S[v][j] for j = 16 w + c (partial over this lane's v)
        // one pass over the value axis (32 values per step): every operand tile
        // is read from LDS once
        // S, dS' rows 32 kp + 4 g + c / 4 (+ 16): the swizzle term is that of
        // row 4 g + c / 4 for every kp
        const int sxo = SXH ? sx_lane_offset(16 * w, g, c) : 0;
#define CARVE_LDSX(B_, R0_) ld_sx_tile<SXH, T, LDSX>(B_, R0_, sxo, 16 * w, g, c)
        for (int kp = 0; kp < NJT / 2; ++kp) {
          CARVE_SEQ();
          const quad s0 = CARVE_LDSX(sSx, 32 * kp);
          const quad s1 = CARVE_LDSX(sSx, 32 * kp + 16);
          const quad a0 = CARVE_LDSX(sdSx, 32 * kp);
          const quad a1 = CARVE_LDSX(sdSx, 32 * kp + 16);
          const quad r0 = CARVE_LDTR(sdRT, LDX, 32 * kp, 0), r1 = CARVE_LDTR(sdRT, LDX, 32 * kp + 16, 0);
          const quad o0 = CARVE_LDTR(sdOT, LDX, 32 * kp, 0), o1 = CARVE_LDTR(sdOT, LDX, 32 * kp + 16, 0);
          const quad u0 = CARVE_LDTR(suT, LDX, 32 * kp, 0), u1 = CARVE_LDTR(suT, LDX, 32 * kp + 16, 0);
          dKt = Qd::mma32(s0, s1, r0, r1, dKt);
          dQt = Qd::mma32(s0, s1, o0, o1, dQt);
          dKi = Qd::mma32(a0, a1, u0, u1, dKi);
          dA = Qd::mma32(r0, r1, u0, u1, dA);
          dP = Qd::mma32(o0, o1, u0, u1, dP);
          // (on the VALU: one more accumulating product here costs the gated
          // kernels registers they do not have)
          const f32x4 x0 = Qd::f32(a0), x1 = Qd::f32(a1), y0 = Qd::f32(s0), y1 = Qd::f32(s1);
          for (int e = 0; e < 4; ++e) dgs += x0[e] * y0[e] + x1[e] * y1[e];
        }
        // the transposed operand tiles of the products after the elementwise
        // gradients, read now: their LDS latency overlaps the permutes below
        const quad KiT = CARVE_LDTR(sKi, LDK, 0, 16 * w);
        const quad KtT = CARVE_LDTR(sKt, LDK, 0, 16 * w), QtT = CARVE_LDTR(sQt, LDK, 0, 16 * w);
        dgs += __shfl_xor(dgs, 16);
        dgs += __shfl_xor(dgs, 32);
        const float bc_ = sBeta[c];
        const f32x4 bq = *reinterpret_cast<const f32x4*>(sBeta + 4 * g);
        const f32x4 gmj = *reinterpret_cast<const f32x4*>(sGam + 16 * w + 4 * g);
        // The factors Kt, Qt, Ki that multiply their gradients in dlam (and Ki in
        // dgam) are the token-dtype values of the operand tiles, exactly as the
        // products above consumed them.  The pair terms of A and P (and the u^T Ki
        // term of the state carry) enter dlam twice with opposite signs and cancel
        // in the suffix sums; with one factor rounded and the other not, the
        // rounding residue of those large terms would not cancel (bf16: about 1 %
        // of dl instead of 0.2 %).
        const int rok = c * LDK + 16 * w + ((4 * g) ^ CARVE_QX(c));
        const f32x4 kiM = Qd::f32(Qd::ld(sKi + rok));
        f32x4 bdA, dgg;
        for (int i = 0; i < 4; ++i) {
          // dgam gam = gam (sum_v dS' S + sum_s Ki_s (dS'^T u_s)), reduced over s = the row
          const float ds = row_scan(kiM[i] * dKi[i]);
          dgg[i] = gmj[i] * (__shfl(dgs, 4 * g + i) + row_bcast15(ds));
          dKt[i] = -bc_ * dKt[i];
          dKi[i] *= gmj[i];
          const bool lowA = c < 4 * g + i, lowP = c <= 4 * g + i;
          dA[i] = lowA ? -dA[i] : 0.0f;
          dP[i] = lowP ? dP[i] : 0.0f;
          bdA[i] = bq[i] * dA[i];
        }
        // beta gradient: A part (dA . A0 summed over s) plus the value partials
        if (w == 0) {
          f32x4 A0 = zero4();
          const T* kr = sKt + c * LDK + ((4 * g) ^ CARVE_QX(c));
          const T* kir = sKi + c * LDK + ((4 * g) ^ CARVE_QX(c));
          for (int jp = 0; jp < NJT / 2; ++jp)
            A0 = Qd::mma32(Qd::ld(kr + 32 * jp), Qd::ld(kr + 32 * jp + 16), Qd::ld(kir + 32 * jp),
                           Qd::ld(kir + 32 * jp + 16), A0);
          // (A0 over the whole tile: its entries above the diagonal are products of
          // factors that may not exist in f32, so they are selected away, not
          // multiplied by the zeros of dA there)
          f32x4 db;
          for (int i = 0; i < 4; ++i) db[i] = row_scan(c < 4 * g + i ? dA[i] * A0[i] : 0.0f);
          // (summed with the value partials by the last wave in the dtau step)
          if (c == 15) *reinterpret_cast<f32x4*>(sDbeta + NW * 16 + 4 * g) = db;
        }
        const quad bdAT = Qd::cvt(Qd::mma16(Qd::cvt(bdA), CARVE_FI(), zero4()));   // rows s, columns t
        const quad dPT = Qd::cvt(Qd::mma16(Qd::cvt(dP), CARVE_FI(), zero4()));
        dKt = Qd::mma16(KiT, bdAT, dKt);
        dKi = Qd::mma32(KtT, QtT, Qd::cvt(bdA), Qd::cvt(dP), dKi);
        dQt = Qd::mma16(KiT, dPT, dQt);
        // elementwise: lane (g, c) holds j = 16 w + 4 g + i, t = c
        f32x4 dzb, dgv, dkv;
        {
        const f32x4 ktM = Qd::f32(Qd::ld(sKt + rok)), qtM = Qd::f32(Qd::ld(sQt + rok));
        for (int i = 0; i < 4; ++i) {
          const float Ep = row_shr1(E[i], row_bcast15(Ei[i]));
          const float nxt = row_shl1(dKt[i] * ktM[i], 0.0f);
          float dlam = dQt[i] * qtM[i] - dKi[i] * kiM[i] + nxt;
          if (c == 15) dlam += dgg[i];
          const float dl = row_suffix(dlam);
          dgv[i] = dl;
          dzb[i] = -dl * sig[i];
          dkv[i] = dKt[i] * Ep + dKi[i] * Ei[i];
          dqp[i] = dQt[i] * E[i];
        }
        }
        Qd::st(dk + e0, Qd::cvt(dkv));
        if constexpr (GATED) {
          // through Eq. decay_gate: df = dg (-exp(A)) sigmoid(f + tau_f); dA and
          // dtau collect dg g and df.  f is read again from its staged tile
          // (the exchange tiles end before it), not kept in registers
          const int byf = (16 * w + 4 * g) * (int)sizeof(T);
          const f32x4 fv = Qd::f32(Qd::ld(sFs + c * D + (((((byf >> 4) ^ (c & (NC - 1))) << 4) | (byf & 15)) / (int)sizeof(T))));
          const f32x4 na = *reinterpret_cast<const f32x4*>(sGate + 16 * w + 4 * g);
          const f32x4 tf = *reinterpret_cast<const f32x4*>(sGate + D + 16 * w + 4 * g);
          f32x4 dfv;
          for (int i = 0; i < 4; ++i) {
            float sp, sg;
            softplus_sigmoid(fv[i] + tf[i], sp, sg);
            dfv[i] = dgv[i] * na[i] * sg;
            gaccA[i] += dgv[i] * na[i] * sp;
            gaccT[i] += dfv[i];
          }
          Qd::st(dfo + e0, Qd::cvt(dfv));
        } else {
          *reinterpret_cast<f32x4*>(dgo + e0) = dgv;
        }
        const quad dzbq = Qd::cvt(dzb);
        Qd::st(dbx + e0, dzbq);
        Qd::st(sdzb + c * LDD + 16 * w + 4 * g, dzbq);
      }
      __syncthreads();

      // -- BT: dtau^T (rows r, column t = c) and dY = dtau (1 - tau^2) -> sdY[t][r]
      for (int x = w; x < (SW ? 1 : 2) * NRB; x += NW) {
        const int rt = x % NRB, side = x / NRB;
        f32x4 acc = zero4();
        if (side == 0) {
          const T* ar = sVbT + (16 * rt + c) * LDK + ((4 * g) ^ CARVE_QX(c));
          const T* br = sdzb + c * LDD + 4 * g;
          for (int jp = 0; jp < NJT / 2; ++jp)
            acc = Qd::mma32(Qd::ld(ar + 32 * jp), Qd::ld(ar + 32 * jp + 16), Qd::ld(br + 32 * jp),
                            Qd::ld(br + 32 * jp + 16), acc);
        } else {
          const T* ar = sVwT + (16 * rt + c) * LDK + ((4 * g) ^ CARVE_QX(c));
          for (int vp = 0; vp < NJT / 2; ++vp)
            acc = Qd::mma32(Qd::ld(ar + 32 * vp), Qd::ld(ar + 32 * vp + 16), CARVE_LDTR(sdzwT, LDX, 32 * vp, 0),
                            CARVE_LDTR(sdzwT, LDX, 32 * vp + 16, 0), acc);
        }
        const int ro = side * RP + 16 * rt + 4 * g;
        const f32x4 tau = Qd::f32(Qd::ld(sTau + c * LDR + ro));
        for (int i = 0; i < 4; ++i) acc[i] *= 1.0f - tau[i] * tau[i];
        Qd::st(sdY + c * LDR + ro, Qd::cvt(acc));
      }
      // beta gradient: the A part plus the value partials, in that order; and
      // (scalar write gate) the write-logit gradient from its value partials.
      // The last wave has no dtau tile at d = 128.
      if (w == NW - 1 && c == 15) {
        f32x4 db = *reinterpret_cast<const f32x4*>(sDbeta + NW * 16 + 4 * g);
        for (int ww = 0; ww < NW; ++ww) {
          const f32x4 pv = *reinterpret_cast<const f32x4*>(sDbeta + ww * 16 + 4 * g);
          for (int i = 0; i < 4; ++i) db[i] += pv[i];
        }
        for (int i = 0; i < 4; ++i) dbeta[(tb + 4 * g + i) * H] = (T)db[i];
        if constexpr (SW) {
          f32x4 dw = zero4();
          for (int ww = 0; ww < NW; ++ww) {
            const f32x4 pv = *reinterpret_cast<const f32x4*>(sDwx + ww * 16 + 4 * g);
            for (int i = 0; i < 4; ++i) dw[i] += pv[i];
          }
          for (int i = 0; i < 4; ++i) dwx[(tb + 4 * g + i) * H] = (T)dw[i];
        }
      }
      // the value-side step took the state gradient with respect to Sr; with
      // respect to S it carries the factor e^{rho}: applied here before the
      // glue, otherwise at the next block's staging
      if (bc == 0) CARVE_BWD_GAM();
      __syncthreads();

      // BQ of this block runs at the top of the next block (or before the glue)
      pdqp = dqp;
      pqq = qq;
      pe0 = e0;
    }
    if (bc != 0) continue;
    {
    // opaque lane coordinates for the glue as well (its LDS addresses are
    // recomputed here rather than held across the loop)
    int tid_ = tid, g_ = g, c_ = c, w_ = w;
    asm volatile("" : "+v"(tid_), "+v"(g_), "+v"(c_), "+v"(w_));
    const int tid = tid_, g = g_, c = c_, w = w_;
    (void)tid;
    CARVE_BWD_BQ();

    // ---- glue: dS += [Ub; Uw]^T dF; dF is parked in the chunk record for
    // d[Ub; Uw] += dF S_hat^T (carve_bwd_param_kernel).  dF enters the product
    // as a high and a low part so that its f32 accumulation is not rounded away.
    {
      constexpr int LDF = R2 + 4;   // row stride of the dF parts (LDS layout)
      T* sdFh = sdSx;               // [D][LDF]: dF[r][j] stored at (j, r)
      T* sdFl = sdSx + D * LDF;     // [D][LDF]: dF - (dF rounded)
      float* dFr = reinterpret_cast<float*>(const_cast<char*>(rc) + cr.dF);
      __syncthreads();  // every wave is done with sdSx and sdY of the last block
      for (int rt = 0; rt < NRT; ++rt) {
        const quad hi = Qd::cvt(dF[rt]);
        Qd::st(sdFh + (16 * w + c) * LDF + 16 * rt + 4 * g, hi);
        Qd::st(sdFl + (16 * w + c) * LDF + 16 * rt + 4 * g, Qd::cvt(dF[rt] - Qd::f32(hi)));
        // dF parked as [j][r] (a lane holds four consecutive r of one j: one
        // 16-byte store per tile); the d[Ub; Uw] kernel transposes it in LDS
        *reinterpret_cast<f32x4*>(dFr + (size_t)(16 * w + c) * R2 + 16 * rt + 4 * g) = dF[rt];
        dF[rt] = zero4();
      }
      __syncthreads();
      for (int jt = 0; jt < NJT; ++jt) {
        CARVE_SEQ();
        // the tile's dF parts in one batch of LDS reads ahead of its products
        quad fh[R2 / 16], fl[R2 / 16];
        for (int rq = 0; rq < R2 / 16; ++rq) {
          const int o = (16 * jt + c) * LDF + 16 * rq + 4 * g;
          fh[rq] = Qd::ld(sdFh + o);
          fl[rq] = Qd::ld(sdFl + o);
        }
        if constexpr (R2 == 64)
          asm volatile("" : "+v"(fh[0]), "+v"(fh[1]), "+v"(fh[2]), "+v"(fh[3]), "+v"(fl[0]), "+v"(fl[1]), "+v"(fl[2]), "+v"(fl[3]));
        f32x4 acc = dSt[jt];
        for (int rp = 0; rp < R2 / 32; ++rp) {
          acc = Qd::mma32(fh[2 * rp], fh[2 * rp + 1], fU[2 * rp], fU[2 * rp + 1], acc);
          acc = Qd::mma32(fl[2 * rp], fl[2 * rp + 1], fU[2 * rp], fU[2 * rp + 1], acc);
        }
        dSt[jt] = acc;
      }
      // (no barrier: the next block writes sdSx only after its first barrier,
      // and what it stages before that barrier does not overlap the dF parts)
    }
    }
  }  // blocks (reverse)

#undef CARVE_BWD_BQ
#undef CARVE_BWD_GAM
#undef CARVE_QX
#undef CARVE_LDTR
#undef CARVE_LDSX
#undef CARVE_BWD_READY
#undef CARVE_BWD_LOADA
#undef CARVE_BWD_LOADS
#undef CARVE_BWD_LOADF
  if constexpr (GATED) {
    // the lanes' sums over their tokens, reduced over the 16 lanes of a row
    // (all tokens of a block) and written by lane c = 0, one owner per channel
    for (int i = 0; i < 4; ++i) {
      gaccA[i] = row_suffix(gaccA[i]);
      gaccT[i] = row_suffix(gaccT[i]);
    }
    if (c == 0) {
      float* dst = a.partG + (size_t)bh * 2 * D + 16 * w + 4 * g;
      *reinterpret_cast<f32x4*>(dst) = gaccA;
      *reinterpret_cast<f32x4*>(dst + D) = gaccT;
    }
  }
  if (a.dS0) {
    float* dst = a.dS0 + soff + (16 * w + c) * D + 4 * g;
    for (int jt = 0; jt < NJT; ++jt) *reinterpret_cast<f32x4*>(dst + 16 * jt) = dSt[jt];
  }
}

// Chunk recompute and adjoint in one grid of nrec + B*H workgroups.  Roles go
// by arrival: each workgroup draws a ticket from the counter in sync; the first
// nrec tickets recompute, the rest run the adjoint of (batch, head) ticket -
// nrec.  A workgroup with a recompute ticket is already running and never
// waits, so every flag an adjoint workgroup waits for is raised in finite time
// whatever order the hardware dispatches the grid in.  Recompute items are
// taken latest chunk first (the order in which the adjoint needs them): item
// i is chunk nch - 1 - i / (B*H) of (batch, head) i % (B*H).  With lead > 0 a
// recompute workgroup starts that chunk only once the adjoint of its (batch,
// head) has started the chunk lead places before it (a bounded wait: the
// recompute still never waits for long): records are then written shortly
// before they are read, and the recompute's stores do not all come at once.
// Measured at the headline shape, a lead of 3-4 chunks takes the fused
// launch from 2.01 to 1.90 ms; 1 chunk starves the adjoint.
template <typename T, int D, int LW, int RP, int VAR>
__global__ void __launch_bounds__(bwd_threads(D)) __attribute__((amdgpu_waves_per_eu(1, 2)))
carve_bwd_fused_kernel(FwdArgs f, BwdArgs a, int nrec, int* sync, int lead) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int nbh = a.B * a.H, nch = a.T / a.L;
  const int nitems = nbh * nch;
  int* ready = sync;
  if (threadIdx.x == 0)
    reinterpret_cast<int*>(smem)[0] =
        __hip_atomic_fetch_add(sync + sync_ticket(nbh, nch), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int ticket = __builtin_amdgcn_readfirstlane(reinterpret_cast<const int*>(smem)[0]);
  __syncthreads();
  if (ticket < nrec) {
    for (int item = ticket; item < nitems; item += nrec) {
      const int ch = nch - 1 - item / nbh, bh = item % nbh;
      const int row = item / nbh;   // chunks after ch
      if (lead > 0 && row >= lead) {
        if (threadIdx.x == 0) {
          const int* p = sync + sync_adjoint_pos(nbh, nch) + bh;
          for (int n = 0; n < kLeadSpinLimit; ++n) {
            if (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) > row - lead) break;
            __builtin_amdgcn_s_sleep(4);
          }
        }
        __syncthreads();
      }
      rec_chunk<T, D, LW, RP, VAR>(f, bh, ch, smem);
      // every wave's record stores are complete before the barrier; the
      // release store (agent scope) then writes them back for other XCDs
      vm_wait_all();
      __syncthreads();
      if (threadIdx.x == 0)
        __hip_atomic_store(ready + (size_t)bh * nch + ch, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  } else {
    bwd_adjoint<T, D, RP, VAR>(a, ticket - nrec, smem, ready, sync + sync_timeout_word(nbh, nch),
                               sync + sync_adjoint_pos(nbh, nch) + (ticket - nrec));
  }
}

// ---------------------------------------------------------------------------
// host-side launch
// ---------------------------------------------------------------------------
template <typename T, int D, int LW, int RP, int VAR>
static int launch_fused_t(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, hipStream_t stream) {
  constexpr size_t lds = fused_lds<T, D, LW, RP, VAR>();
  if constexpr (lds > kMaxLdsBytes) {
    return CARVE_ERR_UNSUPPORTED;
  } else {
    auto kern = carve_bwd_fused_kernel<T, D, LW, RP, VAR>;
    static bool attr_set = false;  // per instantiation
    if (!attr_set) {
      if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds) != hipSuccess)
        return CARVE_ERR_HIP;
      attr_set = true;
    }
    // the adjoint workgroups take B*H compute units (one workgroup per CU: the
    // LDS layout); the recompute gets the rest, or the whole device first when
    // fewer than a quarter would remain
    const int nbh = a.B * a.H;
    const long long nitems = (long long)nbh * (a.T / a.L);
    long long nrec = cus - nbh;
    if (nrec < cus / 4) nrec = cus;
    if (nrec > nitems) nrec = nitems;
    if (nrec < 1) nrec = 1;
    // pace the recompute only when every workgroup of the grid can be resident
    // at once (one per compute unit), so that the adjoints it follows run
    const int lead = nrec + nbh <= cus ? kRecomputeLead : 0;
    hipLaunchKernelGGL(kern, dim3((unsigned)(nrec + nbh)), dim3(bwd_threads(D)), lds, stream, f, a, (int)nrec, sync,
                       lead);
    return hipGetLastError() == hipSuccess ? CARVE_OK : CARVE_ERR_HIP;
  }
}

template <typename T, int D, int RP, int VAR>
static int launch_fused_l(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int LW, hipStream_t s) {
  if (LW == 16) return launch_fused_t<T, D, 16, RP, VAR>(f, a, sync, cus, s);
  if (LW == 32) return launch_fused_t<T, D, 32, RP, VAR>(f, a, sync, cus, s);
  return CARVE_ERR_UNSUPPORTED;
}

template <typename T, int VAR>
static int launch_fused_d(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int D, int LW, hipStream_t s) {
  if (a.RP == 32) {
    if (D == 32) return launch_fused_l<T, 32, 32, VAR>(f, a, sync, cus, LW, s);
    if (D == 64) return launch_fused_l<T, 64, 32, VAR>(f, a, sync, cus, LW, s);
    if (D == 128) return launch_fused_l<T, 128, 32, VAR>(f, a, sync, cus, LW, s);
  } else if (a.RP == 64) {
    if (D == 32) return launch_fused_l<T, 32, 64, VAR>(f, a, sync, cus, LW, s);
    if (D == 64) return launch_fused_l<T, 64, 64, VAR>(f, a, sync, cus, LW, s);
    if (D == 128) return launch_fused_l<T, 128, 64, VAR>(f, a, sync, cus, LW, s);
  }
  return CARVE_ERR_UNSUPPORTED;
}

template <int VAR>
int launch_bwd_fused_var(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int dtype, int D, int LW,
                         hipStream_t s) {
  if (dtype == CARVE_BF16) return launch_fused_d<bf16_t, VAR>(f, a, sync, cus, D, LW, s);
  return launch_fused_d<float, VAR>(f, a, sync, cus, D, LW, s);
}

}  // namespace carve
