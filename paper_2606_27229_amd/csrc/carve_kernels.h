// carve_kernels.h -- kernel argument blocks, LDS layouts and launch entry
// points shared by the CARVE HIP translation units.
#pragma once
#include "../../include/carve.h"
#include "carve_dev.h"

namespace carve {

// ---- forward ----------------------------------------------------------------
struct FwdArgs {
  const void *q, *k, *v, *beta, *bx, *wx;   // token tensors (dtype of the call)
  const float *g, *Ub, *Uw, *Vb, *Vw, *S0;  // f32
  void* o;
  float *S_T, *S_chunks;
  int B, T, H, R, RP, L;
};

// threads of a forward workgroup: one wave per 16-wide tile of the key (and
// value) axis
__host__ __device__ constexpr int fwd_threads(int D) { return (D / 16) * 64; }
// threads of a backward workgroup: one wave per 16-column tile of the state
__host__ __device__ constexpr int bwd_threads(int D) { return (D / 16) * 64; }

__host__ __device__ constexpr size_t lds_round(size_t x) { return (x + 15) & ~(size_t)15; }
__host__ __device__ constexpr size_t lds_max(size_t a, size_t b) { return a > b ? a : b; }

// Token contractions (K = LW) run over LK = max(LW, K per MFMA) columns; the
// padding columns are kept at zero.
template <typename T, int LW>
__host__ __device__ constexpr int lk_of() {
  return (sizeof(T) == 2 && LW < 32) ? 32 : LW;
}

// Forward LDS layout for one sub-chunk of LW tokens (NB = LW / 16 blocks).
// Every row is padded by 16 bytes.  Region X holds the bf16 copy of the chunk
// start state while the fold runs and the per-token key-side operands after.
struct FwdLds {
  size_t U, Q, F, Tau, Beta, X, S, Kt, Qt, Ki, Gam, AT, Tm, P, total;
};

template <typename T, int D, int LW, int RP>
__host__ __device__ constexpr FwdLds fwd_lds() {
  FwdLds l{};
  const size_t e = sizeof(T);
  constexpr size_t NB = LW / 16;
  constexpr size_t PAD = 16 / sizeof(T);
  constexpr size_t LDD = D + PAD, LDR = 2 * RP + PAD, LDB = 16 + PAD;
  size_t off = 0;
  l.U = off;    off += lds_round(2 * RP * LDD * e);
  l.Q = off;    off += lds_round(LW * LDD * e);
  l.F = off;    off += lds_round(2 * RP * LDD * e);
  l.Tau = off;  off += lds_round(LW * LDR * e);
  l.Beta = off; off += lds_round(LW * 4);
  l.X = off;
  size_t x = 0;
  l.Kt = off + x;  x += lds_round(LW * LDD * e);
  l.Qt = off + x;  x += lds_round(LW * LDD * e);
  l.Ki = off + x;  x += lds_round(LW * LDD * e);
  l.Gam = off + x; x += lds_round(NB * D * 4);
  l.AT = off + x;  x += lds_round(NB * 16 * 20 * 4);
  l.Tm = off + x;  x += lds_round(NB * 16 * LDB * e);
  l.P = off + x;   x += lds_round(NB * 16 * LDB * e);
  l.S = off;
  x = lds_max(x, lds_round(D * LDD * e));
  off += x;
  l.total = off;
  return l;
}

int launch_fwd(const FwdArgs& a, int dtype, int D, int LW, hipStream_t s);
size_t fwd_lds_bytes(int dtype, int D, int LW, int RP);

// ---- backward -----------------------------------------------------------------
struct BwdArgs {
  const void *q, *k, *v, *beta, *bx, *wx;
  const float *g, *Ub, *Uw, *Vb, *Vw;
  const float* S_chunks;
  const void* dO;
  const float* dS_T;
  void *dq, *dk, *dv, *dbeta, *dbx, *dwx;
  float* dg;
  float* dS0;
  float* part;       // per-(b,h) partial parameter gradients (workspace)
  float* substates;  // per-(b,h) WY-tile start states inside one gate chunk (workspace)
  const void* Up;    // [2RP][D] packed [Ub; Uw] (token dtype, workspace)
  const void* UT;    // [D][2RP] its transpose (token dtype, workspace)
  int B, T, H, R, RP, L;
};

int launch_bwd(const BwdArgs& a, int dtype, int D, int LW, hipStream_t s);
size_t bwd_lds_bytes(int dtype, int D, int LW, int RP);
int launch_param_reduce(const float* part, int nparts, int R, int D, float* dUb, float* dUw,
                        float* dVb, float* dVw, hipStream_t s);

// size of one per-(b,h) partial-gradient record: dUb, dUw [R][D], dVb, dVw [D][R]
__host__ __device__ constexpr size_t part_floats(int R, int D) { return (size_t)4 * R * D; }

}  // namespace carve
