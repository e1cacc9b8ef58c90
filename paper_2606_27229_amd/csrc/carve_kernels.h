// carve_kernels.h -- kernel argument blocks, LDS layouts and launch entry
// points shared by the CARVE HIP translation units.
#pragma once
#include "../../include/carve.h"
#include "carve_dev.h"

namespace carve {

// Kernel variants (template argument VAR, a bit set):
//   kVarGated:   the decay g is formed in the kernels from its raw logit f
//                (Eq. decay_gate: g = -exp(A) softplus(f + tau_f));
//   kVarScalarW: the scalar write gate (Sec. scalar write gate): one logit wx
//                per (token, head), w = sigmoid(wx) on every value channel and
//                no content term on the write side, so the fold is F = Ub S_hat
//                (R rows instead of 2R) and there is no Uw, Vw;
//   kVarAct:     q, k, v are the raw projections; the kernels apply the input
//                activations (Sec. input projections, Fig. carve_block): q, k =
//                SiLU then L2 normalisation over d_k, v = SiLU.
// Built: every combination of kVarGated and kVarScalarW, and kVarAct alone.
enum : int { kVarGated = 1, kVarScalarW = 2, kVarAct = 4 };
__host__ __device__ constexpr bool var_built(int var) { return var >= 0 && var <= kVarAct; }

// rows of the fold F (and columns of tau) of a variant, R padded to RP:
// [Ub; 0; Uw; 0], or [Ub; 0] with the scalar write gate
__host__ __device__ constexpr int fold_rows(int RP, int var) { return (var & kVarScalarW) ? RP : 2 * RP; }

// ---- forward ----------------------------------------------------------------
struct FwdArgs {
  const void *q, *k, *v, *beta, *bx, *wx;   // token tensors (dtype of the call);
                                            // wx is [B,T,H] with the scalar write gate
  const float *g, *Ub, *Uw, *Vb, *Vw, *S0;  // f32 (Uw, Vw unused with the scalar write gate)
  // decay gate from its raw logit (gated kernels; Eq. decay_gate): f [B,T,H,Dk]
  // in the token dtype, A and tau_f [H,Dk] f32; g is unused then
  const void* f;
  const float *A, *tau_f;
  void* o;
  float *S_T, *S_chunks;
  void* rec;     // chunk records (recompute mode of the backward)
  int B, T, H, R, RP, L;
};

// Per-(batch, head, chunk) record written by the chunk-parallel recompute of
// the backward and read by its adjoint kernel (byte offsets, 256-aligned); RF
// is the variant's number of fold rows (fold_rows):
//   F   [RF][D]    token dtype   folded read-out of the chunk start state
//   Tau [L][RF]    token dtype   tanh(q F^T)
//   Tm  [L/16][16][16]           T = (I + A)^{-1} of every 16-token block
//   P   [L/16][16][16]           P of every block
//   S   [L/16][D/16][threads][4]  block start states scaled by the block's reference,
//                                 Sr = S diag(e^{rho}) with rho = lam_15 / 2 per key
//                                 channel: quad jt of thread tid
//                                 (Sr[16 w + c][16 jt + 4 g + e]), contiguous over threads
//   E   [L/16][16][D]  f32       e^{lam_t - rho} of every token and key channel (its
//                                 block's reference; not written by the GATED kernels)
//   Sig [L/16][16][D]  token dtype  sigma(z_b) of every token and key channel (the
//                                 erase gate b; not written by the GATED kernels)
//   dF  [D][RF]    f32           written by the adjoint: the chunk's gradient of F,
//                                 stored transposed (dF[r][j] at (j, r))
struct ChunkRec {
  size_t F, Tau, Tm, P, S, E, Sig, dF, total;
};
__host__ __device__ constexpr size_t rec_align(size_t x) { return (x + 255) & ~(size_t)255; }
__host__ __device__ constexpr ChunkRec chunk_rec(size_t e, int D, int L, int RF) {
  ChunkRec r{};
  const size_t nbc = L / 16;
  size_t off = 0;
  r.F = off;   off += rec_align((size_t)RF * D * e);
  r.Tau = off; off += rec_align((size_t)L * RF * e);
  r.Tm = off;  off += rec_align(nbc * 256 * e);
  r.P = off;   off += rec_align(nbc * 256 * e);
  r.S = off;   off += rec_align(nbc * (size_t)D * D * e);
  r.E = off;   off += rec_align(nbc * 16 * (size_t)D * 4);
  r.Sig = off; off += rec_align(nbc * 16 * (size_t)D * e);
  r.dF = off;  off += rec_align((size_t)RF * D * 4);
  r.total = off;
  return r;
}

// threads of a forward workgroup: one wave per 16-wide tile of the key (and
// value) axis
__host__ __device__ constexpr int fwd_threads(int D) { return (D / 16) * 64; }
// threads of a backward workgroup: one wave per 16-column tile of the state
__host__ __device__ constexpr int bwd_threads(int D) { return (D / 16) * 64; }

// LDS per workgroup on gfx950
constexpr size_t kMaxLdsBytes = 160 * 1024;

__host__ __device__ constexpr size_t lds_round(size_t x) { return (x + 15) & ~(size_t)15; }
__host__ __device__ constexpr size_t lds_max(size_t a, size_t b) { return a > b ? a : b; }

// Token contractions (K = LW) run over LK = max(LW, K per MFMA) columns; the
// padding columns are kept at zero.
template <typename T, int LW>
__host__ __device__ constexpr int lk_of() {
  return (sizeof(T) == 2 && LW < 32) ? 32 : LW;
}

// LDS layout of the chunk recompute for one sub-chunk of LW tokens (NB = LW / 16
// blocks); SW: the scalar write gate (RP fold rows instead of 2RP).  Every row is padded by 16 bytes.  Region X holds
// the copy of the chunk start state while the fold runs and the per-token
// key-side operands after.  Beta holds beta, then the scalar write gates.
// Kn (kVarAct) holds per-wave partial sums of the squared activated keys.
struct RecLds {
  size_t U, Q, F, Tau, Beta, X, S, Kt, Qt, Ki, Gam, AT, Tm, Gate, Kn, total;
};

template <typename T, int D, int LW, int RP, int VAR>
__host__ __device__ constexpr RecLds rec_lds() {
  RecLds l{};
  const size_t e = sizeof(T);
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr size_t RF = fold_rows(RP, VAR);
  constexpr size_t NB = LW / 16;
  constexpr size_t PAD = 16 / sizeof(T);
  constexpr size_t LDD = D + PAD, LDR = RF + PAD, LDB = 16 + PAD;
  size_t off = 0;
  l.U = off;    off += lds_round(RF * LDD * e);
  l.Q = off;    off += lds_round(LW * LDD * e);
  l.F = off;    off += lds_round(RF * LDD * e);
  l.Tau = off;  off += lds_round(LW * LDR * e);
  l.Beta = off; off += lds_round((SW ? 2 : 1) * LW * 4);
  l.X = off;
  size_t x = 0;
  l.Kt = off + x;  x += lds_round(LW * LDD * e);
  l.Qt = off + x;  x += lds_round(LW * LDD * e);
  l.Ki = off + x;  x += lds_round(LW * LDD * e);
  l.Gam = off + x; x += lds_round(NB * D * 4);
  l.AT = off + x;  x += lds_round(NB * 16 * 20 * 4);
  l.Tm = off + x;  x += lds_round(NB * 16 * LDB * e);
  l.S = off;
  x = lds_max(x, lds_round(D * LDD * e));
  off += x;
  l.Gate = off; off += lds_round(2 * D * 4);   // -exp(A), tau_f of the head (gated)
  l.Kn = off;   off += (VAR & kVarAct) ? lds_round((D / 16) * LW * 4) : 0;
  l.total = off;
  return l;
}

// LDS layout of the chain forward for one WY block of WB tokens (NB = WB / 16
// token tiles); SW: the scalar write gate (RP fold rows instead of 2RP).  Rows
// of n columns take fwd_qstride(n) elements (bf16: 16 (mod 32), the quad
// swizzle qswz; f32: a 16-byte pad).  Region X holds the chunk start
// state while the fold reads it, then the block's raw erase logits (Bx) and the
// decayed keys Kt; Ki holds the block's raw keys until the gates turn them
// into Ki in place.
// With VW (when the layout still fits), VW holds the block's value-side token
// tiles (v, wx: WB rows each, unpadded, 16-byte chunks XOR-swizzled by row) from
// the first barrier of a block to its gates; it overlays A .. TmT, which are
// written only after the gates.  Without VW those tiles are read per wave.
// Tab holds the block's per-channel factor tables, Flag one word per wave
// (whether one of its key channels needs per-tile references).
// Beta holds beta and (scalar write gate) w of the block, for two blocks.
struct ChainLds {
  size_t U, X, Kt, Bx, Ki, F, Q, Tau, A, P, TmT, VW, Tab, Flag, Beta, Gate, total;
};

// Per-channel factor tables of a forward WY block of NB 16-token tiles
// (carve_fwd_chain.h), m_i the reference of tile i and c_i the log retention
// at its end: e^{m_i} (NB rows), e^{lam_end - m_i} (NB), e^{c_i - m_i} (NB),
// e^{lam_end} (1) and e^{m_i - c_j} for i >= j + 2 ((NB - 1) (NB - 2) / 2).  A
// block of one tile needs only e^{m_0}.
// A forward block takes one reference per key channel while every channel's
// log retention over the block stays above -kWideLog (factors up to
// e^{kWideLog / 2}), per-tile references otherwise.
constexpr float kWideLog = 160.0f;
__host__ __device__ constexpr int fwd_tab_rows(int NB) {
  return NB == 1 ? 1 : 3 * NB + 1 + (NB - 1) * (NB - 2) / 2;
}

// Row stride (elements) of a forward operand tile with n columns: bf16 tiles
// take the quad swizzle qswz and need a stride of 16 (mod 32) elements (4 (mod
// 8) quads); f32 tiles keep a 16-byte pad.
template <typename T>
__host__ __device__ constexpr int fwd_qstride(int n) {
  return sizeof(T) == 2 ? (n % 32 == 16 ? n : n + 16) : n + 16 / (int)sizeof(T);
}

template <typename T, int D, int WB, int RP, int VAR, bool VW>
__host__ __device__ constexpr ChainLds chain_lds_v() {
  ChainLds l{};
  const size_t e = sizeof(T);
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr size_t RF = fold_rows(RP, VAR);
  constexpr size_t NB = WB / 16;
  constexpr size_t LDD = fwd_qstride<T>(D), LDR = fwd_qstride<T>(RF), LDW = fwd_qstride<T>(WB),
                   LDB = fwd_qstride<T>(16);
  size_t off = 0;
  l.U = off;    off += lds_round(RF * LDD * e);
  l.X = off;    off += lds_round(lds_max(D * LDD * e, 2 * lds_round(WB * LDD * e)));
  l.Kt = l.X;
  l.Bx = l.X + lds_round(WB * LDD * e);
  l.Ki = off;   off += lds_round(WB * LDD * e);
  l.F = off;    off += lds_round(RF * LDD * e);
  l.Q = off;    off += lds_round(WB * LDD * e);
  l.Tau = off;  off += lds_round(WB * LDR * e);
  l.A = off;    off += lds_round(WB * LDW * e);
  l.P = off;    off += lds_round(WB * LDW * e);
  l.TmT = off;  off += lds_round(NB * 16 * LDB * e);
  l.VW = l.A;
  if (VW) off = lds_max(off, l.VW + lds_round(2 * WB * (size_t)D * e));
  l.Tab = off;  off += lds_round((size_t)fwd_tab_rows((int)NB) * D * 4);
  l.Flag = off; off += lds_round(16 * 4);   // one word per wave
  l.Beta = off; off += lds_round((SW ? 4 : 2) * WB * 4);
  l.Gate = off; off += lds_round(2 * D * 4);   // -exp(A), tau_f of the head (gated)
  l.total = off;
  return l;
}

// whether the value-side tiles are staged (the layout with VW fits)
template <typename T, int D, int WB, int RP, int VAR>
__host__ __device__ constexpr bool chain_stage_vw() {
  return chain_lds_v<T, D, WB, RP, VAR, true>().total <= kMaxLdsBytes;
}

template <typename T, int D, int WB, int RP, int VAR>
__host__ __device__ constexpr ChainLds chain_lds() {
  return chain_lds_v<T, D, WB, RP, VAR, chain_stage_vw<T, D, WB, RP, VAR>()>();
}

// forward of the whole sequence (one workgroup per (batch, head)), WY blocks of
// WB tokens; launch_chain_fwd dispatches on var to launch_chain_fwd_var<VAR>
// (each variant is compiled in a translation unit of its own)
int launch_chain_fwd(const FwdArgs& a, int dtype, int D, int WB, int var, hipStream_t s);
template <int VAR>
int launch_chain_fwd_var(const FwdArgs& a, int dtype, int D, int WB, hipStream_t s);
// LDS bytes of the chain forward of the default variant (2RP fold rows)
size_t chain_lds_bytes(int dtype, int D, int WB, int RP);


// ---- backward -----------------------------------------------------------------
struct BwdArgs {
  const void *q, *k, *v, *beta, *bx, *wx;   // wx (and dwx) [B,T,H] with the scalar write gate
  const float *g, *Ub, *Uw, *Vb, *Vw;
  const float* S_chunks;
  const void* dO;
  const float* dS_T;
  void *dq, *dk, *dv, *dbeta, *dbx, *dwx;
  float* dg;
  // gated kernels: decay logit and its parameters, df (token dtype) instead of
  // dg, per-(b,h) partial dA, dtau ([B*H][2][Dk] f32, workspace)
  const void* f;
  const float *A, *tau_f;
  void* df;
  float* partG;
  float* dS0;
  float* part;    // per-(b,h, chunk split) partial d[Ub; Uw] (workspace)
  float* partV;   // per-(b,h,split) partial dVb, dVw (workspace)
  const void* rec;  // chunk records of the recompute (workspace)
  int B, T, H, R, RP, L;
  int wait_limit;   // polls of the adjoint's bounded wait for a chunk record
};

// token splits of the Vb / Vw gradient kernel and chunk splits of the [Ub; Uw]
// gradient kernel (per (batch, head))
constexpr int kVSplit = 16;
constexpr int kUSplit = 16;

// LDS layout of the adjoint kernel (one 16-token block at a time); SW: the
// scalar write gate (RP fold rows instead of 2RP, no Vw).  The four [value][token]
// exchange buffers dOT .. dzwT are dead between the end of one block and the
// value-side step of the next; the block's token tiles (k, q, bx, v, dO and,
// unless the write gate is scalar, wx, in the token dtype, then g in f32: 16
// rows each, unpadded, 16-byte chunks XOR-swizzled by row) are staged there
// (Stage), so the region holds at least 6 (5) * 16 * D elements plus 16 * D
// floats.  Except in gated kernels, the bx and g slots hold the block's erase
// gate and retention factors E from the chunk record instead.  At a chunk start the glue reuses dSx for dF as a high and a low
// part ([D][LDF] each).
// Gated kernels stage the decay logit f (token dtype) in place of g and keep
// -exp(A), tau_f of the head (Gate) behind it, inside the area g would take
// where that is large enough.  Beta holds beta, then the scalar write gates;
// Dwx the per-wave partial sums of the scalar write gate's gradient.
// Inv (kVarAct) holds the inverse L2 norms of the block's activated keys and
// queries.
struct BwdLds {
  size_t F, VbT, VwT, Tau, Tm, P, Gam, Beta, Dbeta, Dwx, Inv, Kt, Qt, Ki, Sx, dSx, dOT, uT, dRT, dzwT, Stage,
      Gate, dzb, dY, total;
};

// token tiles the adjoint stages per block
__host__ __device__ constexpr int bwd_stage_tiles(bool SW) { return SW ? 5 : 6; }

// Whether the adjoint lays its bf16 operand tiles out bank-conflict-free (the
// quad swizzle qswz).  Not in the gated kernel with the per-channel write
// gate: its extra live state leaves no registers for the swizzle's address
// terms (they raise its spills and cost more than the conflicts they remove).
template <typename T, int VAR>
__host__ __device__ constexpr bool bwd_qswz() {
  return sizeof(T) == 2 && (VAR & (kVarGated | kVarScalarW)) != kVarGated;
}
// Row strides (elements): Kt, Qt, Ki, VbT, VwT (the quad swizzle needs a stride
// of 4 (mod 8) quads; otherwise a 16-byte pad) ...
template <typename T, int D, int VAR>
__host__ __device__ constexpr int bwd_ldk() { return bwd_qswz<T, VAR>() ? D + 16 : D + 16 / (int)sizeof(T); }
// ... the [value][token] exchange tiles ...
template <typename T, int VAR>
__host__ __device__ constexpr int bwd_ldx() { return bwd_qswz<T, VAR>() ? 16 : 16 + 16 / (int)sizeof(T); }
// ... and S, dS' of the block: unpadded rows with the hswz128 swizzle at
// bf16 d = 128, padded rows otherwise
template <typename T, int D, int VAR>
__host__ __device__ constexpr bool bwd_sx_hswz() { return bwd_qswz<T, VAR>() && D == 128; }
template <typename T, int D, int VAR>
__host__ __device__ constexpr int bwd_ldsx() { return bwd_sx_hswz<T, D, VAR>() ? D : D + 16 / (int)sizeof(T); }

template <typename T, int D, int RP, int VAR>
__host__ __device__ constexpr BwdLds bwd_lds() {
  BwdLds l{};
  const size_t e = sizeof(T);
  constexpr bool SW = (VAR & kVarScalarW) != 0;
  constexpr size_t RF = fold_rows(RP, VAR);
  constexpr size_t NW = D / 16;
  constexpr size_t PAD = 16 / sizeof(T);
  constexpr size_t LDD = D + PAD, LDR = RF + PAD, LDB = 16 + PAD;
  constexpr size_t NS = bwd_stage_tiles(SW);
  size_t off = 0;
  constexpr size_t LDK = bwd_ldk<T, D, VAR>(), LDX = bwd_ldx<T, VAR>(), LDSX = bwd_ldsx<T, D, VAR>();
  l.F = off;     off += lds_round(RF * LDD * e);
  l.VbT = off;   off += lds_round(RP * LDK * e);
  l.VwT = off;   off += lds_round((RF - RP) * LDK * e);
  l.Tau = off;   off += lds_round(16 * LDR * e);
  l.Tm = off;    off += lds_round(16 * LDB * e);
  l.P = off;     off += lds_round(16 * LDB * e);
  l.Gam = off;   off += lds_round(D * 4);
  l.Beta = off;  off += lds_round((SW ? 32 : 16) * 4);
  l.Dbeta = off; off += lds_round((NW + 1) * 16 * 4);   // NW value partials + the A part
  l.Dwx = off;   off += SW ? lds_round(NW * 16 * 4) : 0;
  l.Inv = off;   off += (VAR & kVarAct) ? lds_round(2 * 16 * 4) : 0;
  l.Kt = off;    off += lds_round(16 * LDK * e);
  l.Qt = off;    off += lds_round(16 * LDK * e);
  l.Ki = off;    off += lds_round(16 * LDK * e);
  l.Sx = off;    off += lds_round(D * LDSX * e);
  constexpr size_t LDF = RF + 4;
  l.dSx = off;   off += lds_round(D * lds_max(LDSX, 2 * LDF) * e);
  l.Stage = off;
  l.dOT = off;   off += lds_round(D * LDX * e);
  l.uT = off;    off += lds_round(D * LDX * e);
  l.dRT = off;   off += lds_round(D * LDX * e);
  l.dzwT = off;  off += lds_round(D * LDX * e);
  {
    const size_t garea = l.Stage + lds_round(NS * 16 * D * e);     // g, or f then Gate
    l.Gate = garea + lds_round(16 * D * e);
    off = lds_max(off, garea + lds_max(lds_round(16 * D * 4), lds_round(16 * D * e) + lds_round(2 * D * 4)));
  }
  l.dzb = off;   off += lds_round(16 * LDD * e);
  l.dY = off;    off += lds_round(16 * LDR * e);
  l.total = off;
  return l;
}

// LDS of the fused chunk recompute + adjoint launch
template <typename T, int D, int LW, int RP, int VAR>
__host__ __device__ constexpr size_t fused_lds() {
  return lds_max(rec_lds<T, D, LW, RP, VAR>().total, bwd_lds<T, D, RP, VAR>().total);
}

// Chunk recompute and adjoint in one launch (see carve_bwd.h).  f carries the
// forward inputs, S_chunks and the chunk records (f.rec == a.rec); sync points
// at sync_ints(B * H, T / L) ints of workspace, zeroed by launch_sync_clear
// on the same stream before; cus is the device's compute-unit count.
// launch_bwd_fused dispatches on var to launch_bwd_fused_var<VAR>.
int launch_bwd_fused(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int dtype, int D, int LW,
                     int var, hipStream_t s);
template <int VAR>
int launch_bwd_fused_var(const FwdArgs& f, const BwdArgs& a, int* sync, int cus, int dtype, int D, int LW,
                         hipStream_t s);
// dA[h][j], dtau[h][j] = sums over b (in order) of the per-(b,h) partials
int launch_gate_reduce(const float* partG, int B, int H, int D, float* dA, float* dtau, hipStream_t s);
int launch_sync_clear(int* sync, size_t n, hipStream_t s);
// LDS bytes of the fused launch of the default variant with LW-token
// recompute sub-chunks (2RP fold rows)
size_t bwd_lds_bytes(int dtype, int D, int LW, int RP);
// ints of the synchronisation area: one ready flag per chunk, the ticket
// counter that assigns the workgroup roles, the wait-timeout word (nonzero once
// an adjoint wave's bounded wait for a record ran out), padding, then per
// (batch, head) the adjoint's position (chunks it has started, counted from the
// last), which paces the recompute
__host__ __device__ constexpr size_t sync_ints(size_t nbh, size_t nch) { return nbh * nch + 4 + nbh; }
__host__ __device__ constexpr size_t sync_ticket(size_t nbh, size_t nch) { return nbh * nch; }
__host__ __device__ constexpr size_t sync_timeout_word(size_t nbh, size_t nch) { return nbh * nch + 1; }
__host__ __device__ constexpr size_t sync_adjoint_pos(size_t nbh, size_t nch) { return nbh * nch + 4; }
// default bound of that wait, in polls (carve_bwd.h)
constexpr int kReadySpinLimit = 1 << 20;
// d[Ub; Uw] over chunk splits and dVb, dVw over token splits (carve_param.h),
// one launch; sw: the scalar write gate (dVb, dUb only; the records hold RP
// fold rows)
int launch_bwd_param(const BwdArgs& a, int dtype, int D, bool sw, hipStream_t s);
// in one launch: sum npartU records of 2 * half floats at partU into dU0 (first
// half) and dU1, and npartV records at partV into dV0 and dV1; with dU1 == dV1
// == NULL only the first halves are summed
int launch_param_reduce(const float* partU, int npartU, const float* partV, int npartV, size_t half, float* dU0,
                        float* dU1, float* dV0, float* dV1, hipStream_t s);
// kVarAct: turn dq, dk (gradients of the activated q, k, in place, [rows][D]) into
// the gradients of the raw projections q_raw, k_raw
int launch_act_bwd(const void* q_raw, const void* k_raw, void* dq, void* dk, size_t rows, int D, int dtype,
                   hipStream_t s);

// Output RMS normalisation over rows of N = H * Dv values (carve_norm.hip).
// The backward's workgroups (at most kNormBwdGroups) each write one f32
// partial row of dweight, summed in order by a second launch; mark (if not
// NULL) is called between the two launches.
constexpr int kNormBwdGroups = 1024;
// carve_rmsnorm_bwd_noalloc: bytes of the per-device static scratch (every
// supported row length: kNormBwdGroups partial rows of up to 4096 floats) and
// the devices it can address
constexpr size_t kNormScratchBytes = (size_t)kNormBwdGroups * 4096 * sizeof(float);
constexpr int kMaxNormDevices = 64;
int norm_scratch(float** ptr);
bool rmsnorm_supported(int dtype, int N);
int rmsnorm_bwd_groups(long rows);
int launch_rmsnorm_fwd(const void* x, const float* wt, void* y, long rows, int N, float eps, int dtype,
                       hipStream_t s);
int launch_rmsnorm_bwd(const void* x, const float* wt, const void* dy, void* dx, float* partial, float* dw, long rows,
                       int N, float eps, int dtype, hipStream_t s, void (*mark)(hipStream_t));

// floats of one partial-gradient record: d[Ub; Uw] ([R][D] twice) or dVb, dVw ([D][R] twice)
__host__ __device__ constexpr size_t part_floats(int R, int D) { return (size_t)2 * R * D; }

}  // namespace carve
