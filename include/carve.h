/*
 * carve.h -- C ABI of libcarve: the chunked CARVE layer (arXiv 2606.27229)
 * forward and backward on AMD Instinct MI355X (gfx950).
 *
 * What the library computes (one layer, every batch element b and head h,
 * recurrent state S in R^{Dv x Dk}):
 *
 *   Sec. 4, Eq. carve_state (boxed): per token t
 *       S_t = S_{t-1} diag(exp g_t) diag(1 - b_t) + beta_t (w_t * v_t - S_{t-1} k_t) k_t^T
 *       o_t = S_t q_t
 *     with key-axis decay g_t (log domain, <= 0) and erase gate b_t, a
 *     per-token write strength beta_t, and a value-axis write gate w_t that
 *     scales v_t only (Alg. WYChunkDelta step 3).
 *   Sec. 4.2, Eq. content_readout / erase_gate: the gates of every token of
 *     chunk c (tokens [cL, (c+1)L)) read the state carried out of chunk c-1
 *     (S0 for chunk 0), folded once per chunk:
 *       F = [Ub; Uw] S_{c-1}           (2R x Dk)
 *       tau_b = tanh(F_b q_t), tau_w = tanh(F_w q_t)
 *       b_t = sigmoid(bx_t + Vb tau_b),  w_t = sigmoid(wx_t + Vw tau_w)
 *   Sec. 6.2, Alg. WYChunkDelta: evaluated chunk-parallel in WY form (one
 *     shared unit-lower-triangular solve per chunk, Thm. chunkability).
 *   App. Alg. backward / megakernel_bwd: the exact gradient of
 *       loss = <dO, o> + <dS_T, S_T>
 *     with respect to every input, including the chunk-boundary "glue"
 *     through the folded read-out and the parameter gradients reduced over
 *     batch, heads and chunks.
 *
 * Conventions
 *   - All tensors are dense, row-major and live in DEVICE memory owned by
 *     the caller.  Token tensors are [B, T, H, D] (q, k, bx, g: D = Dk;
 *     v, wx, o: D = Dv); beta is [B, T, H]; states are [B, H, Dv, Dk];
 *     S_chunks is [B, H, T/L, Dv, Dk] and holds the state at the start of
 *     every chunk; Ub, Uw are [R, Dv]; Vb is [Dk, R]; Vw is [Dv, R].
 *     Ub, Uw, Vb, Vw are shared by all heads.
 *   - dtype (CARVE_F32 or CARVE_BF16) is the element type of q, k, v, beta,
 *     bx, wx, o, dO and of dq, dk, dv, dbeta, dbx, dwx.  g, the parameters,
 *     the states and dg, dUb, dUw, dVb, dVw, dS0, dS_T are always f32.  All
 *     arithmetic is f32 (bf16 operands on the matrix cores in bf16 mode).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the
 *     default stream) and never synchronises.  The return value reports
 *     argument validation and launch errors only.
 *   - Outputs are overwritten, never accumulated (parameter gradients too).
 *   - The library allocates no device memory and keeps no state between
 *     calls except the cached kernel attributes; concurrent calls on
 *     different streams must use different workspaces.
 *   - Supported shapes: Dk == Dv in {32, 64, 128}; 1 <= R <= 64;
 *     L in {16, 32, 64, 128}; T a positive multiple of L; B, H >= 1.
 *     Not built (their LDS layouts exceed 160 KB): the forward with f32
 *     token tensors at Dk = 128 and R > 32; the backward with f32 token
 *     tensors at Dk = 128, and with R > 32 at Dk = 128 (bf16) or Dk = 64
 *     (f32).  These, and other shapes, return CARVE_ERR_UNSUPPORTED
 *     (CARVE_ERR_SHAPE when T % L != 0 or a size is non-positive).
 *   - Every pointer must be 16-byte aligned (CARVE_ERR_ALIGN).
 *   - Inputs are assumed finite with g <= 0; NaN/Inf propagate.  Numerical
 *     range (log retention l = g - softplus(z_b) per key channel): the
 *     forward evaluates WY blocks of up to 64 tokens; a key channel whose
 *     sum of l over a block stays above -160 is taken relative to the middle
 *     of that block's range, any other channel relative to the middle of
 *     each 16-token tile's range, with the products across tiles formed from
 *     operands no larger than the raw token values.  The sum of l over every
 *     16-token tile must stay above about -150 (-170 where a block is a
 *     single tile).  The backward evaluates 16-token blocks relative to the
 *     middle of their range, with factors up to e^{|sum of l over the block|
 *     / 2}, so each such block must sum above about -170.
 */
#ifndef CARVE_H
#define CARVE_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { CARVE_F32 = 0, CARVE_BF16 = 1 } carve_dtype_t;

typedef struct {
  int B, T, H, Dk, Dv, R, L;
  carve_dtype_t dtype;
} carve_dims_t;

enum {
  CARVE_OK = 0,
  CARVE_ERR_NULL = -1,        /* a required pointer is NULL */
  CARVE_ERR_SHAPE = -2,       /* non-positive size or T % L != 0 */
  CARVE_ERR_UNSUPPORTED = -3, /* valid but not built: see "Supported shapes" */
  CARVE_ERR_ALIGN = -4,       /* a pointer is not 16-byte aligned */
  CARVE_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than carve_workspace_size */
  CARVE_ERR_HIP = -6,         /* a HIP runtime call failed */
  CARVE_ERR_ARG = -7          /* conflicting or invalid argument values (g and f both given; eps) */
};

/* Bytes of device workspace the forward (for_backward = 0) or the backward
 * (for_backward = 1) needs for these dims; 0 means none.  Returns 0 for
 * dims that fail validation.  The workspace holds the per-chunk records of
 * the recompute (fold, tau, WY factors and block start states), the partial
 * parameter gradients and the chunk ready flags of the fused recompute +
 * adjoint launch (the same size for the gated backward). */
size_t carve_workspace_size(const carve_dims_t* d, int for_backward);

/* Forward (Alg. carve_fwd with the WY solve of Alg. WYChunkDelta).
 * In:  q, k [B,T,H,Dk]; v [B,T,H,Dv]; beta [B,T,H]; g [B,T,H,Dk] (f32);
 *      bx [B,T,H,Dk]; wx [B,T,H,Dv]; Ub, Uw, Vb, Vw (f32);
 *      S0 [B,H,Dv,Dk] f32 or NULL (= zeros).
 * Out: o [B,T,H,Dv]; S_T [B,H,Dv,Dk] or NULL; S_chunks [B,H,T/L,Dv,Dk] or
 *      NULL (needed by carve_chunk_bwd).
 * workspace may be NULL when carve_workspace_size(d, 0) == 0. */
int carve_chunk_fwd(const carve_dims_t* d, const void* q, const void* k, const void* v,
                    const void* beta, const float* g, const void* bx, const void* wx,
                    const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                    const float* S0, void* o, float* S_T, float* S_chunks, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* Backward of carve_chunk_fwd for loss <dO, o> + <dS_T, S_T>.
 * In:  the forward inputs; S_chunks as written by carve_chunk_fwd on the
 *      same inputs; dO [B,T,H,Dv]; dS_T [B,H,Dv,Dk] f32 or NULL (= zeros).
 * Out: dq, dk [B,T,H,Dk]; dv [B,T,H,Dv]; dbeta [B,T,H]; dg [B,T,H,Dk] f32;
 *      dbx [B,T,H,Dk]; dwx [B,T,H,Dv]; dUb, dUw [R,Dv]; dVb [Dk,R];
 *      dVw [Dv,R]; dS0 [B,H,Dv,Dk] or NULL.  (S0 itself is not needed: the
 *      chunk-start states are read from S_chunks.)
 * The parameter gradients are reduced over batch, heads and chunks in a
 * fixed order, so reruns are bitwise identical. */
int carve_chunk_bwd(const carve_dims_t* d, const void* q, const void* k, const void* v,
                    const void* beta, const float* g, const void* bx, const void* wx,
                    const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                    const float* S_chunks, const void* dO, const float* dS_T, void* dq, void* dk,
                    void* dv, void* dbeta, float* dg, void* dbx, void* dwx, float* dUb,
                    float* dUw, float* dVb, float* dVw, float* dS0, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* The same layer with the key-axis decay computed from its raw logit inside
 * the kernels (Sec. decay_gate, Eq. decay_gate: "gate-in-kernel" fusion):
 *     g[b,t,h,j] = -exp(A[h][j]) * softplus(f[b,t,h,j] + tau_f[h][j])
 * In:  f [B,T,H,Dk] in the call's dtype (the raw decay logit, replacing g);
 *      A, tau_f [H,Dk] f32: learned log-amplitudes and biases of the gate
 *      (tau_f is the bias the paper calls tau in Eq. decay_gate, not the
 *      content read-out tau of Eq. content_readout); the other arguments are
 *      those of carve_chunk_fwd.  g is never materialised.
 * The numerical-range precondition applies to the g so formed. */
int carve_chunk_fwd_gated(const carve_dims_t* d, const void* q, const void* k, const void* v,
                          const void* beta, const void* f, const float* A, const float* tau_f,
                          const void* bx, const void* wx, const float* Ub, const float* Uw,
                          const float* Vb, const float* Vw, const float* S0, void* o, float* S_T,
                          float* S_chunks, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Backward of carve_chunk_fwd_gated for loss <dO, o> + <dS_T, S_T>.  Outputs
 * as carve_chunk_bwd, with dg replaced by:
 *   df [B,T,H,Dk] in the call's dtype: dL/df = dL/dg * (-exp(A)) * sigmoid(f + tau_f);
 *   dA, dtau [H,Dk] f32: sums over batch and tokens of dL/dg * g and of dL/df,
 *   reduced in a fixed order (bitwise-reproducible reruns).
 * The workspace is the one carve_workspace_size(d, 1) reports. */
int carve_chunk_bwd_gated(const carve_dims_t* d, const void* q, const void* k, const void* v,
                          const void* beta, const void* f, const float* A, const float* tau_f,
                          const void* bx, const void* wx, const float* Ub, const float* Uw,
                          const float* Vb, const float* Vw, const float* S_chunks, const void* dO,
                          const float* dS_T, void* dq, void* dk, void* dv, void* dbeta, void* df,
                          float* dA, float* dtau, void* dbx, void* dwx, float* dUb, float* dUw,
                          float* dVb, float* dVw, float* dS0, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* The layer with the scalar write gate (Sec. scalar write gate, the deployment
 * variant of the ablation rows "scalar write" of Table attribution): one write
 * logit per token and head, broadcast over the value channels, and no content
 * term on the write side:
 *     w_t = sigmoid(wx[b,t,h]) on every one of the Dv channels,
 *     b_t = sigmoid(bx_t + Vb tanh(F_b q_t)) with F_b = Ub S_{c-1} (as before).
 * The fold has R rows instead of 2R; there is no Uw, Vw.
 * In:  wx [B,T,H] in the call's dtype (replacing the [B,T,H,Dv] logits);
 *      the decay either as g [B,T,H,Dk] f32 (f = A = tau_f = NULL) or from its
 *      raw logit as in carve_chunk_fwd_gated (g = NULL; f, A, tau_f given);
 *      the other arguments are those of carve_chunk_fwd.
 * Returns CARVE_ERR_NULL when neither g nor f is given, CARVE_ERR_ARG when
 * both are.  Ub = 0 gives the ablation's row with no content at all. */
int carve_chunk_fwd_sw(const carve_dims_t* d, const void* q, const void* k, const void* v,
                       const void* beta, const float* g, const void* f, const float* A,
                       const float* tau_f, const void* bx, const void* wx, const float* Ub,
                       const float* Vb, const float* S0, void* o, float* S_T, float* S_chunks,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Backward of carve_chunk_fwd_sw for loss <dO, o> + <dS_T, S_T>.  Outputs as
 * carve_chunk_bwd (dg with the g form; df, dA, dtau as carve_chunk_bwd_gated
 * with the f form; the other decay outputs may be NULL), except:
 *   dwx [B,T,H] in the call's dtype: the sum over the value channels of the
 *   per-channel write-logit gradient, dL/dwx_t = sum_v dL/dw_tv * w_t (1 - w_t);
 *   no dUw, dVw.
 * The workspace is the one carve_workspace_size(d, 1) reports; the launch
 * sequence (and the measurement hook's events) is that of the matching
 * carve_chunk_bwd or carve_chunk_bwd_gated call. */
int carve_chunk_bwd_sw(const carve_dims_t* d, const void* q, const void* k, const void* v,
                       const void* beta, const float* g, const void* f, const float* A,
                       const float* tau_f, const void* bx, const void* wx, const float* Ub,
                       const float* Vb, const float* S_chunks, const void* dO, const float* dS_T,
                       void* dq, void* dk, void* dv, void* dbeta, float* dg, void* df, float* dA,
                       float* dtau, void* dbx, void* dwx, float* dUb, float* dVb, float* dS0,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The layer with its input activations inside the kernels (Sec. input
 * projections, Fig. carve_block, the chunk-local normalisation of
 * Alg. megakernel fused into the chunk loads):
 *     q = SiLU(q_raw) / sqrt(|SiLU(q_raw)|^2 + 1e-6)   per (token, head) over Dk,
 *     k likewise from k_raw, v = SiLU(v_raw).
 * In:  q, k, v are the raw projections q_raw, k_raw, v_raw (same shapes and
 *      dtype as in carve_chunk_fwd); every other argument is that of
 *      carve_chunk_fwd.  The activated q, k, v are never written to memory. */
int carve_chunk_fwd_act(const carve_dims_t* d, const void* q, const void* k, const void* v,
                        const void* beta, const float* g, const void* bx, const void* wx,
                        const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                        const float* S0, void* o, float* S_T, float* S_chunks, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* Backward of carve_chunk_fwd_act for loss <dO, o> + <dS_T, S_T>.  Outputs as
 * carve_chunk_bwd, with dq, dk, dv the gradients with respect to q_raw, k_raw,
 * v_raw.  The backward makes one more launch than carve_chunk_bwd (the last:
 * dq, dk taken through the L2 normalisation and SiLU in place). */
int carve_chunk_bwd_act(const carve_dims_t* d, const void* q, const void* k, const void* v,
                        const void* beta, const float* g, const void* bx, const void* wx,
                        const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                        const float* S_chunks, const void* dO, const float* dS_T, void* dq, void* dk,
                        void* dv, void* dbeta, float* dg, void* dbx, void* dwx, float* dUb,
                        float* dUw, float* dVb, float* dVw, float* dS0, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* Output RMS normalisation, the step that closes Alg. carve_fwd:
 *     y = W_O RMSNorm(reshape(o)),
 * without W_O (a plain GEMM outside the recurrence).  Alg. megakernel runs it
 * as one hoisted launch over the assembled o, and Alg. megakernel_bwd mirrors
 * it with one hoisted launch of its gradient; these entry points are those
 * launches.  A token's row is reshape(o)[b, t, :], the N = H * Dv values of
 * all its heads ([B, T, H, Dv] row-major viewed as [B*T, N]):
 *     y[row, i] = o[row, i] / sqrt(mean_i o[row, i]^2 + eps) * weight[i]
 * The paper gives no eps; the Python binding passes 1e-6.
 * Only B, T, H, Dv and dtype of d are read (Dk, R and L are not; T need not be
 * a multiple of L).  Supported: N a multiple of 8 (bf16) or 4 (f32) with
 * N <= 4096 (bf16) or 2048 (f32), else CARVE_ERR_UNSUPPORTED; eps finite and
 * >= 0, else CARVE_ERR_ARG.  A row of zeros with eps = 0 gives NaN.
 * In:  o [B,T,H,Dv] in the call's dtype (as written by carve_chunk_fwd);
 *      weight [H*Dv] f32.
 * Out: y [B,T,H,Dv] in the call's dtype (must not overlap o or weight).
 * One launch; asynchronous on stream. */
int carve_rmsnorm_fwd(const carve_dims_t* d, const void* o, const float* weight, float eps, void* y,
                      hipStream_t stream);

/* Bytes of device workspace carve_rmsnorm_bwd needs for these dims (one f32
 * partial row of dweight per workgroup of its first launch, at most 1024);
 * 0 for dims that fail validation. */
size_t carve_rmsnorm_workspace_size(const carve_dims_t* d);

/* Backward of carve_rmsnorm_fwd for loss <dy, y>:
 *     r = 1 / sqrt(mean_i o_i^2 + eps),  n = o r,  dn = dy * weight,
 *     d_o = r (dn - n mean_i(dn_i n_i)),  dweight = sum over rows of dy * n.
 * In:  o, weight, eps as given to the forward; dy [B,T,H,Dv] in the call's dtype.
 * Out: d_o [B,T,H,Dv] in the call's dtype; dweight [H*Dv] f32 (overwritten,
 *      reduced over the rows in a fixed order: reruns are bitwise identical).
 * workspace: at least carve_rmsnorm_workspace_size(d) bytes, else
 * CARVE_ERR_WORKSPACE.  Two launches (the rows, then the fixed-order sum of
 * the workgroups' dweight partials); no output may overlap an input or the
 * workspace. */
int carve_rmsnorm_bwd(const carve_dims_t* d, const void* o, const float* weight, float eps, const void* dy,
                      void* d_o, float* dweight, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* carve_rmsnorm_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It allocates nothing: the dweight
 * partials go to a static device array of the library, 16 MiB (1024 partial
 * rows of up to 4096 floats), which every supported shape fits; each GPU the
 * library runs on holds its own copy until the process ends.  Its device
 * address is looked up once per device, on the first call made with that
 * device current (CARVE_ERR_HIP if the lookup fails).  Arguments, outputs and
 * errors are those of carve_rmsnorm_bwd; the results are bitwise those of
 * carve_rmsnorm_bwd.  Every call on one GPU shares that GPU's array: calls
 * that overlap in time on one GPU (different streams, or different threads
 * without ordering) race on it and must not be made. */
int carve_rmsnorm_bwd_noalloc(const carve_dims_t* d, const void* o, const float* weight, float eps,
                              const void* dy, void* d_o, float* dweight, hipStream_t stream);

/* Measurement hook (not part of the computation).  Arms the next
 * carve_chunk_* or carve_rmsnorm_* call made on the calling thread to record
 * events[0] on its stream before its first kernel launch and events[i] after
 * its i-th launch (the forward makes 1 launch; the backward 6: clear of the
 * chunk ready flags, chunk recompute fused with the adjoint, dVb/dVw
 * partials, d[Ub;Uw] partials, two fixed-order reductions; the gated backward
 * a 7th, the reduction of dA, dtau over the batch; the backward with the
 * input activations a 7th, the activation gradient of dq, dk; the norm's
 * forward 1, its backward 2),
 * up to `capacity` events.  `events` are hipEvent_t handles created by the
 * caller (hipEventCreate) and owned by the caller; the handles are copied
 * here (the array may be freed after this call) and the events are only
 * recorded, never synchronised.  The hook covers exactly one call and is
 * cleared when that call returns, whatever its status; capacity 0 disarms
 * it.  Returns CARVE_ERR_NULL for a NULL array with capacity > 0 or a
 * negative capacity, CARVE_ERR_UNSUPPORTED for capacity > 16. */
int carve_profile_events(hipEvent_t* events, int capacity);

/* Diagnostic of the backward's wait for the chunk records (not part of the
 * computation).  In carve_chunk_bwd and its variants, each adjoint wave waits
 * for the records of the next chunks with a bounded poll of their ready flags
 * (by default 2^20 polls, about a second; a correct launch never reaches it,
 * since a chunk is recomputed in tens of microseconds by a workgroup that is
 * already running).  If the bound runs out, the wave fills its state gradient
 * with NaN, so the gradients of all earlier tokens come out NaN, waits no
 * more, and sets a timeout word in the workspace's synchronisation area.  The
 * call itself still returns CARVE_OK, as kernel completion is asynchronous.
 * This reads that word for the last backward enqueued with `workspace` and
 * the same dims `d`: *timed_out = 1 if a wait ran out, 0 otherwise.  The word
 * is cleared at the start of every backward.  It copies 4 bytes to the host on
 * `stream` and synchronises `stream`: the only call of this library that
 * synchronises.  Errors: CARVE_ERR_NULL for a NULL argument;
 * CARVE_ERR_SHAPE / CARVE_ERR_UNSUPPORTED for dims no backward accepts;
 * CARVE_ERR_HIP if the copy fails. */
int carve_bwd_wait_status(const carve_dims_t* d, const void* workspace, hipStream_t stream, int* timed_out);

/* Test hook for the timeout path above: sets the bound of that wait, in polls,
 * for the backward calls made on the calling thread from then on.  0 makes
 * every wait give up at once (the kernels still run to completion and the
 * results are NaN); a negative value restores the default.  Returns the
 * previous bound.  Not for production use. */
int carve_set_ready_wait_limit(int polls);

/* Static description of a status code. */
const char* carve_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* CARVE_H */
