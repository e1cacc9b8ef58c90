/*
 * carve_oracle.h -- CPU reference (oracle) for the chunked CARVE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this library: only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header or constant with the
 * HIP implementation.
 *
 * Everything is double precision on host memory.  Layouts (row-major):
 *   q, k, bx, g : [B, T, H, Dk]      v, wx, o : [B, T, H, Dv]
 *   beta        : [B, T, H]
 *   Ub, Uw      : [R, Dv]  (erase / write down-projections W_{U1,b}, W_{U1,w})
 *   Vb          : [Dk, R]  (erase up-projection W_{U2,b})
 *   Vw          : [Dv, R]  (write up-projection W_{U2,w})
 *   S0, S_T     : [B, H, Dv, Dk]     S_chunks : [B, H, T/L, Dv, Dk]
 * The parameters Ub, Uw, Vb, Vw are shared by every head.
 *
 * Return value: 0 on success, -1 on a NULL required pointer, -2 on a shape
 * error (non-positive sizes or T % L != 0).
 */
#ifndef CARVE_ORACLE_H
#define CARVE_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int B, T, H, Dk, Dv, R, L;
} cref_dims;

/* Token-serial definition (Sec. 4, Eq. carve_state with the gates of
 * Eq. content_readout / erase_gate evaluated on the chunk-boundary state).
 * S0 may be NULL (zeros).  S_T, S_chunks, gate_b [B,T,H,Dk], gate_w [B,T,H,Dv]
 * may be NULL.  nthreads <= 0 means one thread. */
int cref_fwd_serial(const cref_dims* d, const double* q, const double* k, const double* v,
                    const double* beta, const double* g, const double* bx, const double* wx,
                    const double* Ub, const double* Uw, const double* Vb, const double* Vw,
                    const double* S0, double* o, double* S_T, double* S_chunks,
                    double* gate_b, double* gate_w, int nthreads);

/* The same layer in chunked WY form (Sec. 6.2, Alg. WYChunkDelta, Eq.
 * gamma_cum / M_coupling), written with plain loops and an explicit
 * forward substitution.  Same arguments as cref_fwd_serial. */
int cref_fwd_chunked(const cref_dims* d, const double* q, const double* k, const double* v,
                     const double* beta, const double* g, const double* bx, const double* wx,
                     const double* Ub, const double* Uw, const double* Vb, const double* Vw,
                     const double* S0, double* o, double* S_T, double* S_chunks,
                     double* gate_b, double* gate_w, int nthreads);

/* Memory-blind key-axis gated delta recurrence: b = sigmoid(bx),
 * w = sigmoid(wx), no state readout (Sec. 4.2, zero-initialised content
 * projections).  Written independently of the two functions above. */
int cref_baseline_fwd(const cref_dims* d, const double* q, const double* k, const double* v,
                      const double* beta, const double* g, const double* bx, const double* wx,
                      const double* S0, double* o, double* S_T, int nthreads);

/* Exact reverse mode of cref_fwd_serial (App. Alg. backward, re-derived).
 * The loss is <dO, o> + <dS_T, S_T>; dS_T may be NULL (zeros), S0 may be
 * NULL.  All gradient outputs are overwritten.  dS0 may be NULL. */
int cref_bwd(const cref_dims* d, const double* q, const double* k, const double* v,
             const double* beta, const double* g, const double* bx, const double* wx,
             const double* Ub, const double* Uw, const double* Vb, const double* Vw,
             const double* S0, const double* dO, const double* dS_T,
             double* dq, double* dk, double* dv, double* dbeta, double* dg,
             double* dbx, double* dwx, double* dUb, double* dUw, double* dVb,
             double* dVw, double* dS0, int nthreads);

/* Key-axis decay gate from its raw logit (Sec. decay_gate, Eq. decay_gate):
 * g[b,t,h,j] = -exp(A[h][j]) * softplus(f[b,t,h,j] + tau[h][j]).
 * f, g : [B, T, H, Dk];  A, tau : [H, Dk]. */
int cref_decay_gate(const cref_dims* d, const double* f, const double* A, const double* tau, double* g);

/* Its reverse mode: df [B,T,H,Dk] = dg * (-exp(A) sigmoid(f + tau));
 * dA [H,Dk] = sum over b, t of dg * g;  dtau [H,Dk] = sum over b, t of df. */
int cref_decay_gate_bwd(const cref_dims* d, const double* f, const double* A, const double* tau,
                        const double* dg, double* df, double* dA, double* dtau);

#ifdef __cplusplus
}
#endif
#endif
