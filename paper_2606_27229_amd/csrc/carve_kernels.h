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

struct FwdLds {
  size_t S, Q, K, Ki, F, Tau, KhT, A, Base, Cf, Beta, Ucat, Vb, Vw, total;
};

// threads of a forward workgroup: up to four waves (one per SIMD)
__host__ __device__ constexpr int fwd_threads(int D) { return (D / 16 < 4 ? D / 16 : 4) * 64; }
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

template <typename T, int D, int LW>
__host__ __device__ constexpr FwdLds fwd_lds(int RP) {
  FwdLds l{};
  size_t off = 0;
  const size_t e = sizeof(T);
  constexpr int NB = LW / 16;
  constexpr int LK = lk_of<T, LW>();
  constexpr size_t PAD = 16 / sizeof(T);      // every LDS row is padded by 16 bytes
  constexpr size_t LDD = D + PAD, LDK = LK + PAD, LDA = LW + 4;
  const size_t LDR = 2 * (size_t)RP + PAD, LDV = (size_t)RP + PAD;
  l.S = off;    off += lds_round((size_t)D * LDD * e);
  l.Q = off;    off += lds_round(lds_max((size_t)LW * LDD, (size_t)D * LDK) * e);   // also R^T [D][LK]
  l.K = off;    off += lds_round(lds_max((size_t)LW * LDD, (size_t)D * LDK) * e);   // also u^T [D][LK]
  l.Ki = off;   off += lds_round(lds_max((size_t)LW * LDD, (size_t)LW * LDK) * e);  // also P [LW][LK]
  l.F = off;    off += lds_round((size_t)2 * RP * LDD * e);
  l.Tau = off;  off += lds_round(lds_max((size_t)LW * LDR, (size_t)LW * LDK) * e);  // also T [LW][LK]
  l.KhT = off;  off += lds_round((size_t)D * LDK * e);
  l.A = off;    off += lds_round((size_t)LW * LDA * 4);
  l.Base = off; off += lds_round((size_t)NB * D * 4);
  l.Cf = off;   off += lds_round((size_t)NB * NB * D * 4);
  l.Beta = off; off += lds_round((size_t)LW * 4);
  l.Ucat = off; off += lds_round((size_t)2 * RP * LDD * e);
  l.Vb = off;   off += lds_round((size_t)D * LDV * e);
  l.Vw = off;   off += lds_round((size_t)D * LDV * e);
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
