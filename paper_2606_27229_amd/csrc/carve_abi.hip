// carve_abi.hip -- the C ABI of libcarve: argument validation, workspace
// sizing, kernel selection and launch.  No allocation, no synchronisation.
#include <stdint.h>

#include "carve_kernels.h"

using namespace carve;

namespace {

constexpr size_t kMaxLds = 160 * 1024;

int round_rp(int R) { return (R + 31) / 32 * 32; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// backward workspace: d[Ub; Uw] partials per (b,h, chunk split) | dVb, dVw
// partials per (b,h, token split) | chunk records of the recompute | ready
// flags and ticket counter of the fused recompute + adjoint launch
struct BwdWs {
  size_t part, partV, rec, sync, partG, total;
};

BwdWs bwd_workspace_layout(const carve_dims_t* d) {
  BwdWs l{};
  const size_t nbh = (size_t)d->B * d->H;
  const size_t es = d->dtype == CARVE_BF16 ? 2 : 4;
  const size_t nch = (size_t)(d->T / d->L);
  size_t off = 0;
  l.part = off;  off += align256(nbh * kUSplit * part_floats(d->R, d->Dk) * 4);
  l.partV = off; off += align256(nbh * kVSplit * part_floats(d->R, d->Dk) * 4);
  // records of the full layer (2RP fold rows); the scalar-write records are smaller
  l.rec = off;   off += align256(nbh * nch * chunk_rec(es, d->Dk, d->L, 2 * round_rp(d->R)).total);
  l.sync = off;  off += align256(sync_ints(nbh, nch) * sizeof(int));
  l.partG = off; off += align256(nbh * 2 * (size_t)d->Dk * 4);   // dA, dtau partials (gated)
  l.total = off;
  return l;
}

size_t esize(carve_dtype_t dt) { return dt == CARVE_BF16 ? 2 : 4; }

int check_dims(const carve_dims_t* d) {
  if (!d) return CARVE_ERR_NULL;
  if (d->B <= 0 || d->T <= 0 || d->H <= 0 || d->Dk <= 0 || d->Dv <= 0 || d->R <= 0 || d->L <= 0)
    return CARVE_ERR_SHAPE;
  if (d->dtype != CARVE_F32 && d->dtype != CARVE_BF16) return CARVE_ERR_UNSUPPORTED;
  if (d->T % d->L != 0) return CARVE_ERR_SHAPE;
  if (d->Dk != d->Dv) return CARVE_ERR_UNSUPPORTED;
  if (d->Dk != 32 && d->Dk != 64 && d->Dk != 128) return CARVE_ERR_UNSUPPORTED;
  if (d->R > 64) return CARVE_ERR_UNSUPPORTED;
  if (d->L != 16 && d->L != 32 && d->L != 64 && d->L != 128) return CARVE_ERR_UNSUPPORTED;
  // the grid is B*H workgroups; inside one (batch, head) the kernels address
  // token tensors with 32-bit offsets
  if ((long long)d->B * d->H > (1LL << 30)) return CARVE_ERR_UNSUPPORTED;
  if ((long long)d->T * d->H * (d->Dk > d->Dv ? d->Dk : d->Dv) >= (1LL << 31)) return CARVE_ERR_UNSUPPORTED;
  return CARVE_OK;
}

// largest recompute sub-chunk (<= 32 tokens, dividing L) for which the LDS
// layout of the fused recompute + adjoint launch fits.  32-token sub-chunks
// keep the recompute's registers within the file (64-token ones spill 64 of
// them) and recompute fastest: measured against 64 and 16 tokens, the fused
// launch took 1.32 against 1.49 and 1.41 ms at B = 8, H = 16, T = 2048 (where
// the recompute bounds it) and 1.885 against 1.90 and 1.884 ms at the
// 1.3B-scale T = 4096 layer (where the adjoint does)
int pick_lw(const carve_dims_t* d) {
  const int RP = round_rp(d->R);
  for (int lw = 32; lw >= 16; lw /= 2) {
    if (lw > d->L || d->L % lw) continue;
    if (bwd_lds_bytes(d->dtype, d->Dk, lw, RP) <= kMaxLds) return lw;
  }
  return 0;
}

// compute units of the current device (the fused backward sizes its grid by it)
int device_cus(int* cus) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CARVE_ERR_HIP;
  if (hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return CARVE_ERR_HIP;
  if (*cus < 1) *cus = 1;
  return CARVE_OK;
}

// largest WY block (<= 64 tokens, dividing L) whose chain-forward LDS layout fits
int pick_wb(const carve_dims_t* d) {
  const int RP = round_rp(d->R);
  for (int wb = 64; wb >= 16; wb /= 2) {
    if (wb > d->L || d->L % wb) continue;
    if (chain_lds_bytes(d->dtype, d->Dk, wb, RP) <= kMaxLds) return wb;
  }
  return 0;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// launch-boundary events of the next call on this thread (carve_profile_events);
// the handles are copied when the hook is armed
constexpr int kMaxProfEvents = 16;
thread_local hipEvent_t g_prof_events[kMaxProfEvents];
thread_local int g_prof_capacity = 0;
thread_local int g_prof_count = 0;

void prof_mark(hipStream_t stream) {
  if (g_prof_count < g_prof_capacity) hipEventRecord(g_prof_events[g_prof_count++], stream);
}

// the hook covers exactly one call: it is cleared when that call returns,
// whatever its status
struct ProfClear {
  ~ProfClear() { g_prof_capacity = 0; }
};

// bound of the backward's wait for a chunk record, for the calls made on this
// thread (carve_set_ready_wait_limit)
thread_local int g_wait_limit = kReadySpinLimit;

struct Range {
  const void* p;
  size_t bytes;
};

bool overlap(const Range& a, const Range& b) {
  if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes, b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
  return a0 < b1 && b0 < a1;
}

bool any_overlap(const Range* outs, int nout, const Range* ins, int nin) {
  for (int i = 0; i < nout; ++i) {
    for (int j = 0; j < nin; ++j)
      if (overlap(outs[i], ins[j])) return true;
    for (int j = i + 1; j < nout; ++j)
      if (overlap(outs[i], outs[j])) return true;
  }
  return false;
}

}  // namespace

extern "C" {

const char* carve_status_string(int status) {
  switch (status) {
    case CARVE_OK: return "ok";
    case CARVE_ERR_NULL: return "a required pointer is NULL";
    case CARVE_ERR_SHAPE: return "invalid shape (non-positive size or T not a multiple of L)";
    case CARVE_ERR_UNSUPPORTED: return "unsupported configuration (dtype, head size, rank or chunk length)";
    case CARVE_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case CARVE_ERR_WORKSPACE: return "workspace missing or too small";
    case CARVE_ERR_HIP: return "HIP runtime error";
    case CARVE_ERR_ARG: return "conflicting or invalid argument values (both of two alternative inputs given, or eps)";
    default: return "unknown status";
  }
}

int carve_profile_events(hipEvent_t* events, int capacity) {
  g_prof_capacity = 0;
  if (capacity < 0 || (capacity > 0 && !events)) return CARVE_ERR_NULL;
  if (capacity > kMaxProfEvents) return CARVE_ERR_UNSUPPORTED;
  for (int i = 0; i < capacity; ++i) g_prof_events[i] = events[i];
  g_prof_capacity = capacity;
  g_prof_count = 0;
  return CARVE_OK;
}

int carve_set_ready_wait_limit(int polls) {
  const int prev = g_wait_limit;
  g_wait_limit = polls < 0 ? kReadySpinLimit : polls;
  return prev;
}

int carve_bwd_wait_status(const carve_dims_t* d, const void* workspace, hipStream_t stream, int* timed_out) {
  if (!d || !workspace || !timed_out) return CARVE_ERR_NULL;
  int st = check_dims(d);
  if (st) return st;
  if (!pick_lw(d)) return CARVE_ERR_UNSUPPORTED;
  const BwdWs wl = bwd_workspace_layout(d);
  const int* word = reinterpret_cast<const int*>(reinterpret_cast<const char*>(workspace) + wl.sync) +
                    sync_timeout_word((size_t)d->B * d->H, (size_t)(d->T / d->L));
  int h = 0;
  if (hipMemcpyAsync(&h, word, sizeof(int), hipMemcpyDeviceToHost, stream) != hipSuccess) return CARVE_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return CARVE_ERR_HIP;
  *timed_out = h != 0 ? 1 : 0;
  return CARVE_OK;
}

size_t carve_workspace_size(const carve_dims_t* d, int for_backward) {
  if (check_dims(d) != CARVE_OK) return 0;
  if (!for_backward) return 0;
  if (!pick_lw(d)) return 0;
  return bwd_workspace_layout(d).total;
}

}  // extern "C"

namespace {

// the decay input: g itself, or its raw logit f with A, tau_f (Eq. decay_gate)
struct Decay {
  const float* g;
  const void* f;
  const float *A, *tau_f;
  bool gated() const { return f != nullptr; }
};

// kernel variant of a call
int variant_of(const Decay& dc, bool sw, bool act) {
  return (dc.gated() ? kVarGated : 0) | (sw ? kVarScalarW : 0) | (act ? kVarAct : 0);
}

// sw: the scalar write gate (wx [B,T,H], no Uw, Vw); act: q, k, v are the raw
// projections (the kernels apply the input activations)
int fwd_impl(const carve_dims_t* d, const void* q, const void* k, const void* v, const void* beta,
             const Decay& dc, const void* bx, const void* wx, const float* Ub, const float* Uw,
             const float* Vb, const float* Vw, const float* S0, void* o, float* S_T, float* S_chunks,
             bool sw, bool act, hipStream_t stream) {
  ProfClear pc;
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !bx || !wx || !Ub || !Vb || !o) return CARVE_ERR_NULL;
  if (!sw && (!Uw || !Vw)) return CARVE_ERR_NULL;
  if (dc.gated() ? (!dc.A || !dc.tau_f) : !dc.g) return CARVE_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, dc.g, dc.f, dc.A, dc.tau_f, bx, wx, Ub, Uw, Vb, Vw, S0, o, S_T, S_chunks};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return CARVE_ERR_ALIGN;
  const size_t es = esize(d->dtype);
  const size_t ntok = (size_t)d->B * d->T * d->H;
  const size_t nst = (size_t)d->B * d->H * d->Dv * d->Dk;
  const size_t HD = (size_t)d->H * d->Dk * 4;
  const Range ins[] = {{q, ntok * d->Dk * es}, {k, ntok * d->Dk * es}, {v, ntok * d->Dv * es},
                       {beta, ntok * es}, {dc.g, ntok * d->Dk * 4}, {dc.f, ntok * d->Dk * es},
                       {dc.A, HD}, {dc.tau_f, HD}, {bx, ntok * d->Dk * es},
                       {wx, ntok * (sw ? 1 : d->Dv) * es}, {Ub, (size_t)d->R * d->Dv * 4},
                       {Uw, (size_t)d->R * d->Dv * 4}, {Vb, (size_t)d->Dk * d->R * 4},
                       {Vw, (size_t)d->Dv * d->R * 4}, {S0, nst * 4}};
  const Range outs[] = {{o, ntok * d->Dv * es}, {S_T, nst * 4}, {S_chunks, nst * (d->T / d->L) * 4}};
  if (any_overlap(outs, 3, ins, 15)) return CARVE_ERR_UNSUPPORTED;
  const int wb = pick_wb(d);
  if (!wb) return CARVE_ERR_UNSUPPORTED;
  FwdArgs a;
  a.q = q; a.k = k; a.v = v; a.beta = beta; a.bx = bx; a.wx = wx;
  a.g = dc.g; a.Ub = Ub; a.Uw = Uw; a.Vb = Vb; a.Vw = Vw; a.S0 = S0;
  a.f = dc.f; a.A = dc.A; a.tau_f = dc.tau_f;
  a.o = o; a.S_T = S_T; a.S_chunks = S_chunks;
  a.B = d->B; a.T = d->T; a.H = d->H; a.R = d->R; a.RP = round_rp(d->R); a.L = d->L;
  a.rec = nullptr;
  prof_mark(stream);
  st = launch_chain_fwd(a, d->dtype, d->Dk, wb, variant_of(dc, sw, act), stream);
  prof_mark(stream);
  return st;
}

// decay gradient: dg, or df with dA, dtau (gated)
struct DecayGrad {
  float* dg;
  void* df;
  float *dA, *dtau;
};

int bwd_impl(const carve_dims_t* d, const void* q, const void* k, const void* v, const void* beta,
             const Decay& dc, const void* bx, const void* wx, const float* Ub, const float* Uw,
             const float* Vb, const float* Vw, const float* S_chunks, const void* dO, const float* dS_T,
             void* dq, void* dk, void* dv, void* dbeta, const DecayGrad& dd, void* dbx, void* dwx,
             float* dUb, float* dUw, float* dVb, float* dVw, float* dS0, void* workspace,
             size_t workspace_bytes, bool sw, bool act, hipStream_t stream) {
  ProfClear pc;
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !bx || !wx || !Ub || !Vb || !S_chunks || !dO ||
      !dq || !dk || !dv || !dbeta || !dbx || !dwx || !dUb || !dVb)
    return CARVE_ERR_NULL;
  if (!sw && (!Uw || !Vw || !dUw || !dVw)) return CARVE_ERR_NULL;
  if (dc.gated() ? (!dc.A || !dc.tau_f || !dd.df || !dd.dA || !dd.dtau) : (!dc.g || !dd.dg)) return CARVE_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, dc.g, dc.f, dc.A, dc.tau_f, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO, dS_T,
                        dq, dk, dv, dbeta, dd.dg, dd.df, dd.dA, dd.dtau, dbx, dwx, dUb, dUw, dVb, dVw, dS0,
                        workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return CARVE_ERR_ALIGN;
  const size_t need = carve_workspace_size(d, 1);
  if (need && (!workspace || workspace_bytes < need)) return CARVE_ERR_WORKSPACE;
  const size_t es = esize(d->dtype);
  const size_t ntok = (size_t)d->B * d->T * d->H;
  const size_t nst = (size_t)d->B * d->H * d->Dv * d->Dk;
  const size_t RDv = (size_t)d->R * d->Dv * 4;
  const size_t HD = (size_t)d->H * d->Dk * 4;
  const size_t nwx = ntok * (sw ? 1 : d->Dv) * es;   // bytes of wx and of dwx
  const Range ins[] = {{q, ntok * d->Dk * es}, {k, ntok * d->Dk * es}, {v, ntok * d->Dv * es},
                       {beta, ntok * es}, {dc.g, ntok * d->Dk * 4}, {dc.f, ntok * d->Dk * es},
                       {dc.A, HD}, {dc.tau_f, HD}, {bx, ntok * d->Dk * es},
                       {wx, nwx}, {Ub, RDv}, {Uw, RDv}, {Vb, RDv}, {Vw, RDv},
                       {S_chunks, nst * (d->T / d->L) * 4}, {dO, ntok * d->Dv * es},
                       {dS_T, nst * 4}, {workspace, need}};
  const Range outs[] = {{dq, ntok * d->Dk * es}, {dk, ntok * d->Dk * es}, {dv, ntok * d->Dv * es},
                        {dbeta, ntok * es}, {dd.dg, ntok * d->Dk * 4}, {dd.df, ntok * d->Dk * es},
                        {dd.dA, HD}, {dd.dtau, HD}, {dbx, ntok * d->Dk * es},
                        {dwx, nwx}, {dUb, RDv}, {dUw, RDv}, {dVb, RDv},
                        {dVw, RDv}, {dS0, nst * 4}};
  if (any_overlap(outs, 15, ins, 18)) return CARVE_ERR_UNSUPPORTED;
  const int lw = pick_lw(d);
  if (!lw) return CARVE_ERR_UNSUPPORTED;
  int cus = 0;
  st = device_cus(&cus);
  if (st) return st;
  const BwdWs wl = bwd_workspace_layout(d);
  char* wsb = reinterpret_cast<char*>(workspace);
  const int RP = round_rp(d->R);
  // 1-2. chunk-parallel recompute -> chunk records, overlapped with the adjoint
  FwdArgs f;
  f.q = q; f.k = k; f.v = v; f.beta = beta; f.bx = bx; f.wx = wx;
  f.g = dc.g; f.Ub = Ub; f.Uw = Uw; f.Vb = Vb; f.Vw = Vw; f.S0 = nullptr;
  f.f = dc.f; f.A = dc.A; f.tau_f = dc.tau_f;
  f.o = nullptr; f.S_T = nullptr; f.S_chunks = const_cast<float*>(S_chunks);
  f.rec = wsb + wl.rec;
  f.B = d->B; f.T = d->T; f.H = d->H; f.R = d->R; f.RP = RP; f.L = d->L;
  BwdArgs a;
  a.q = q; a.k = k; a.v = v; a.beta = beta; a.bx = bx; a.wx = wx;
  a.g = dc.g; a.Ub = Ub; a.Uw = Uw; a.Vb = Vb; a.Vw = Vw; a.S_chunks = S_chunks;
  a.f = dc.f; a.A = dc.A; a.tau_f = dc.tau_f;
  a.dO = dO; a.dS_T = dS_T;
  a.dq = dq; a.dk = dk; a.dv = dv; a.dbeta = dbeta; a.dbx = dbx; a.dwx = dwx; a.dg = dd.dg; a.dS0 = dS0;
  a.df = dd.df;
  a.part = reinterpret_cast<float*>(wsb + wl.part);
  a.partV = reinterpret_cast<float*>(wsb + wl.partV);
  a.partG = reinterpret_cast<float*>(wsb + wl.partG);
  a.rec = wsb + wl.rec;
  a.B = d->B; a.T = d->T; a.H = d->H; a.R = d->R; a.RP = RP; a.L = d->L;
  a.wait_limit = g_wait_limit;
  int* sync = reinterpret_cast<int*>(wsb + wl.sync);
  prof_mark(stream);
  st = launch_sync_clear(sync, sync_ints((size_t)d->B * d->H, (size_t)(d->T / d->L)), stream);
  if (st) return st;
  prof_mark(stream);
  st = launch_bwd_fused(f, a, sync, cus, d->dtype, d->Dk, lw, variant_of(dc, sw, act), stream);
  if (st) return st;
  prof_mark(stream);
  // 3. in one launch: d[Ub; Uw] from the per-chunk dF, dVb, dVw from dbx, dwx
  //    and tau (dUb, dVb only with the scalar write gate)
  st = launch_bwd_param(a, d->dtype, d->Dk, sw, stream);
  if (st) return st;
  prof_mark(stream);
  // 4. fixed-order reductions of the partials
  const int nbh = d->B * d->H;
  const size_t RD = (size_t)d->R * d->Dk;
  st = launch_param_reduce(a.part, nbh * kUSplit, a.partV, nbh * kVSplit, RD, dUb, sw ? nullptr : dUw, dVb,
                           sw ? nullptr : dVw, stream);
  if (st) return st;
  prof_mark(stream);
  // 5. (gated) dA, dtau summed over the batch
  if (dc.gated()) {
    st = launch_gate_reduce(a.partG, d->B, d->H, d->Dk, dd.dA, dd.dtau, stream);
    if (st) return st;
    prof_mark(stream);
  }
  // 6. (input activations) dq, dk through the L2 normalisation and SiLU
  if (act) {
    st = launch_act_bwd(q, k, dq, dk, (size_t)d->B * d->T * d->H, d->Dk, d->dtype, stream);
    prof_mark(stream);
  }
  return st;
}

}  // namespace

extern "C" {

int carve_chunk_fwd(const carve_dims_t* d, const void* q, const void* k, const void* v,
                    const void* beta, const float* g, const void* bx, const void* wx,
                    const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                    const float* S0, void* o, float* S_T, float* S_chunks, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  return fwd_impl(d, q, k, v, beta, Decay{g, nullptr, nullptr, nullptr}, bx, wx, Ub, Uw, Vb, Vw, S0, o, S_T,
                  S_chunks, false, false, stream);
}

int carve_chunk_fwd_gated(const carve_dims_t* d, const void* q, const void* k, const void* v,
                          const void* beta, const void* f, const float* A, const float* tau_f,
                          const void* bx, const void* wx, const float* Ub, const float* Uw,
                          const float* Vb, const float* Vw, const float* S0, void* o, float* S_T,
                          float* S_chunks, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  if (!f) {
    ProfClear pc;
    return CARVE_ERR_NULL;
  }
  return fwd_impl(d, q, k, v, beta, Decay{nullptr, f, A, tau_f}, bx, wx, Ub, Uw, Vb, Vw, S0, o, S_T, S_chunks,
                  false, false, stream);
}

int carve_chunk_bwd(const carve_dims_t* d, const void* q, const void* k, const void* v,
                    const void* beta, const float* g, const void* bx, const void* wx,
                    const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                    const float* S_chunks, const void* dO, const float* dS_T, void* dq, void* dk,
                    void* dv, void* dbeta, float* dg, void* dbx, void* dwx, float* dUb,
                    float* dUw, float* dVb, float* dVw, float* dS0, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
  return bwd_impl(d, q, k, v, beta, Decay{g, nullptr, nullptr, nullptr}, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO,
                  dS_T, dq, dk, dv, dbeta, DecayGrad{dg, nullptr, nullptr, nullptr}, dbx, dwx, dUb, dUw, dVb,
                  dVw, dS0, workspace, workspace_bytes, false, false, stream);
}

int carve_chunk_bwd_gated(const carve_dims_t* d, const void* q, const void* k, const void* v,
                          const void* beta, const void* f, const float* A, const float* tau_f,
                          const void* bx, const void* wx, const float* Ub, const float* Uw,
                          const float* Vb, const float* Vw, const float* S_chunks, const void* dO,
                          const float* dS_T, void* dq, void* dk, void* dv, void* dbeta, void* df,
                          float* dA, float* dtau, void* dbx, void* dwx, float* dUb, float* dUw,
                          float* dVb, float* dVw, float* dS0, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (!f) {
    ProfClear pc;
    return CARVE_ERR_NULL;
  }
  return bwd_impl(d, q, k, v, beta, Decay{nullptr, f, A, tau_f}, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO, dS_T,
                  dq, dk, dv, dbeta, DecayGrad{nullptr, df, dA, dtau}, dbx, dwx, dUb, dUw, dVb, dVw, dS0,
                  workspace, workspace_bytes, false, false, stream);
}

int carve_chunk_fwd_sw(const carve_dims_t* d, const void* q, const void* k, const void* v,
                       const void* beta, const float* g, const void* f, const float* A,
                       const float* tau_f, const void* bx, const void* wx, const float* Ub,
                       const float* Vb, const float* S0, void* o, float* S_T, float* S_chunks,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  if (!g == !f) {
    ProfClear pc;
    return g ? CARVE_ERR_ARG : CARVE_ERR_NULL;
  }
  const Decay dc = g ? Decay{g, nullptr, nullptr, nullptr} : Decay{nullptr, f, A, tau_f};
  return fwd_impl(d, q, k, v, beta, dc, bx, wx, Ub, nullptr, Vb, nullptr, S0, o, S_T, S_chunks, true, false, stream);
}

int carve_chunk_bwd_sw(const carve_dims_t* d, const void* q, const void* k, const void* v,
                       const void* beta, const float* g, const void* f, const float* A,
                       const float* tau_f, const void* bx, const void* wx, const float* Ub,
                       const float* Vb, const float* S_chunks, const void* dO, const float* dS_T,
                       void* dq, void* dk, void* dv, void* dbeta, float* dg, void* df, float* dA,
                       float* dtau, void* dbx, void* dwx, float* dUb, float* dVb, float* dS0,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!g == !f) {
    ProfClear pc;
    return g ? CARVE_ERR_ARG : CARVE_ERR_NULL;
  }
  const Decay dc = g ? Decay{g, nullptr, nullptr, nullptr} : Decay{nullptr, f, A, tau_f};
  const DecayGrad dd = g ? DecayGrad{dg, nullptr, nullptr, nullptr} : DecayGrad{nullptr, df, dA, dtau};
  return bwd_impl(d, q, k, v, beta, dc, bx, wx, Ub, nullptr, Vb, nullptr, S_chunks, dO, dS_T, dq, dk, dv, dbeta, dd,
                  dbx, dwx, dUb, nullptr, dVb, nullptr, dS0, workspace, workspace_bytes, true, false, stream);
}

int carve_chunk_fwd_act(const carve_dims_t* d, const void* q, const void* k, const void* v,
                        const void* beta, const float* g, const void* bx, const void* wx,
                        const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                        const float* S0, void* o, float* S_T, float* S_chunks, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  return fwd_impl(d, q, k, v, beta, Decay{g, nullptr, nullptr, nullptr}, bx, wx, Ub, Uw, Vb, Vw, S0, o, S_T,
                  S_chunks, false, true, stream);
}

int carve_chunk_bwd_act(const carve_dims_t* d, const void* q, const void* k, const void* v,
                        const void* beta, const float* g, const void* bx, const void* wx,
                        const float* Ub, const float* Uw, const float* Vb, const float* Vw,
                        const float* S_chunks, const void* dO, const float* dS_T, void* dq, void* dk,
                        void* dv, void* dbeta, float* dg, void* dbx, void* dwx, float* dUb,
                        float* dUw, float* dVb, float* dVw, float* dS0, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  return bwd_impl(d, q, k, v, beta, Decay{g, nullptr, nullptr, nullptr}, bx, wx, Ub, Uw, Vb, Vw, S_chunks, dO,
                  dS_T, dq, dk, dv, dbeta, DecayGrad{dg, nullptr, nullptr, nullptr}, dbx, dwx, dUb, dUw, dVb,
                  dVw, dS0, workspace, workspace_bytes, false, true, stream);
}

}  // extern "C"

// ---- output RMS normalisation (Alg. carve_fwd output step, hoisted) --------

namespace {

// rows and row length of reshape(o) [B*T, H*Dv]; only B, T, H, Dv and dtype
// of the dims are read
int norm_dims(const carve_dims_t* d, long* rows, int* N) {
  if (!d) return CARVE_ERR_NULL;
  if (d->B <= 0 || d->T <= 0 || d->H <= 0 || d->Dv <= 0) return CARVE_ERR_SHAPE;
  if (d->dtype != CARVE_F32 && d->dtype != CARVE_BF16) return CARVE_ERR_UNSUPPORTED;
  const long long n = (long long)d->H * d->Dv;
  if (n > (1 << 20) || !rmsnorm_supported(d->dtype, (int)n)) return CARVE_ERR_UNSUPPORTED;
  const long long r = (long long)d->B * d->T;
  if (r * n >= (1LL << 62)) return CARVE_ERR_UNSUPPORTED;
  *rows = (long)r;
  *N = (int)n;
  return CARVE_OK;
}

bool eps_ok(float eps) { return eps >= 0.0f && eps <= 3.0e38f; }   // false for NaN and +Inf

}  // namespace

extern "C" {

size_t carve_rmsnorm_workspace_size(const carve_dims_t* d) {
  long rows = 0;
  int N = 0;
  if (norm_dims(d, &rows, &N) != CARVE_OK) return 0;
  return align256((size_t)rmsnorm_bwd_groups(rows) * N * sizeof(float));
}

int carve_rmsnorm_fwd(const carve_dims_t* d, const void* o, const float* weight, float eps, void* y,
                      hipStream_t stream) {
  ProfClear pc;
  long rows = 0;
  int N = 0;
  int st = norm_dims(d, &rows, &N);
  if (st) return st;
  if (!o || !weight || !y) return CARVE_ERR_NULL;
  if (!eps_ok(eps)) return CARVE_ERR_ARG;
  if (!aligned16(o) || !aligned16(weight) || !aligned16(y)) return CARVE_ERR_ALIGN;
  const size_t es = esize(d->dtype);
  const Range ins[] = {{o, (size_t)rows * N * es}, {weight, (size_t)N * 4}};
  const Range outs[] = {{y, (size_t)rows * N * es}};
  if (any_overlap(outs, 1, ins, 2)) return CARVE_ERR_UNSUPPORTED;
  prof_mark(stream);
  st = launch_rmsnorm_fwd(o, weight, y, rows, N, eps, d->dtype, stream);
  prof_mark(stream);
  return st;
}

int carve_rmsnorm_bwd_noalloc(const carve_dims_t* d, const void* o, const float* weight, float eps, const void* dy,
                              void* d_o, float* dweight, hipStream_t stream) {
  long rows = 0;
  int N = 0;
  int st = norm_dims(d, &rows, &N);
  if (st) {
    ProfClear pc;
    return st;
  }
  const size_t need = carve_rmsnorm_workspace_size(d);
  if (need > kNormScratchBytes) {
    ProfClear pc;
    return CARVE_ERR_WORKSPACE;
  }
  float* ws = nullptr;
  st = norm_scratch(&ws);
  if (st) {
    ProfClear pc;
    return st;
  }
  return carve_rmsnorm_bwd(d, o, weight, eps, dy, d_o, dweight, ws, kNormScratchBytes, stream);
}

int carve_rmsnorm_bwd(const carve_dims_t* d, const void* o, const float* weight, float eps, const void* dy,
                      void* d_o, float* dweight, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  ProfClear pc;
  long rows = 0;
  int N = 0;
  int st = norm_dims(d, &rows, &N);
  if (st) return st;
  if (!o || !weight || !dy || !d_o || !dweight) return CARVE_ERR_NULL;
  if (!eps_ok(eps)) return CARVE_ERR_ARG;
  const void* ptrs[] = {o, weight, dy, d_o, dweight, workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return CARVE_ERR_ALIGN;
  const size_t need = carve_rmsnorm_workspace_size(d);
  if (!workspace || workspace_bytes < need) return CARVE_ERR_WORKSPACE;
  const size_t es = esize(d->dtype);
  const size_t nx = (size_t)rows * N * es;
  const Range ins[] = {{o, nx}, {weight, (size_t)N * 4}, {dy, nx}, {workspace, need}};
  const Range outs[] = {{d_o, nx}, {dweight, (size_t)N * 4}};
  if (any_overlap(outs, 2, ins, 4)) return CARVE_ERR_UNSUPPORTED;
  prof_mark(stream);
  st = launch_rmsnorm_bwd(o, weight, dy, d_o, reinterpret_cast<float*>(workspace), dweight, rows, N, eps, d->dtype,
                          stream, prof_mark);
  prof_mark(stream);
  return st;
}

}  // extern "C"
