// Host side of the C ABI declared in include/rla.h: argument validation (no
// HIP call until it passes), workspace planning and launch sequencing.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "rla.h"

namespace rla {
namespace {

constexpr size_t kAlign = 256;

// Opt-in stage timing (rla_set_stage_events): events recorded on the launch
// stream at the start of a call and after each kernel stage.
thread_local hipEvent_t* g_events = nullptr;
thread_local int g_num_events = 0;
thread_local int g_next_event = 0;

hipError_t mark_stage(hipStream_t stream, bool first) {
  if (first) g_next_event = 0;
  if (!g_events || g_next_event >= g_num_events) return hipSuccess;
  return hipEventRecord(g_events[g_next_event++], stream);
}

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Problem {
  int64_t B = 0, T = 0, H = 0, DK = 0, DV = 0, N = 0, ntok = 0, max_chunks = 0;
  bool varlen = false, bf16 = false, out_bf16 = false, save = false, use_saved = false;
  int32_t vflags = 0;   // kVar* bits
  const float* decay_param = nullptr;
  float* decay_param_grad = nullptr;
  const int32_t* cu = nullptr;
  float clip = -1.f;
};

struct Workspace {
  size_t seqs = 0, chunks = 0, nchunks = 0, order = 0, gates = 0, mats = 0;
  size_t ckS = 0, ckR = 0, mask = 0, dS = 0, dR = 0, fblk = 0, bblk = 0, total = 0;
  size_t ckS_sc = 0, ckR_sc = 0, dS_sc = 0, dR_sc = 0;
  size_t qh = 0, kh = 0, dqh = 0, dkh = 0, dpart = 0;   // pre-processing
  size_t gmax = 0, gscale = 0;   // upstream-gradient maxima and scales (bf16 backward)
};

// recurrent: the decoding step, whose kernel has no fp32 d_k restriction
rla_status check_problem(const rla_problem* pp, Problem& pr, bool recurrent = false) {
  if (!pp) return RLA_ERR_NULL_ARG;
  if (pp->dtype != RLA_F32 && pp->dtype != RLA_BF16) return RLA_ERR_DTYPE;
  if (pp->batch < 0 || pp->seq_len < 0 || pp->num_heads < 1) return RLA_ERR_SHAPE;
  if (pp->num_heads > 65535) return RLA_ERR_SHAPE;
  const bool dk_ok = pp->head_dim_k == 64 || pp->head_dim_k == 128;
  const bool dv_ok = pp->head_dim_v == 64 || pp->head_dim_v == 128;
  if (!dk_ok || !dv_ok) return RLA_ERR_SHAPE;
  if (!recurrent && pp->dtype == RLA_F32 && pp->head_dim_k != 64) return RLA_ERR_DTYPE;
  if (pp->out_dtype != RLA_F32 && pp->out_dtype != RLA_BF16) return RLA_ERR_DTYPE;
  if (pp->dtype == RLA_F32 && pp->out_dtype != RLA_F32) return RLA_ERR_DTYPE;
  if (isnan(pp->clip) || pp->clip < 0.f) return RLA_ERR_VALUE;
  constexpr uint32_t kKnown = RLA_FLAG_SAVE_FOR_BACKWARD | RLA_FLAG_USE_SAVED |
                              RLA_FLAG_RESIDUAL_TANH | RLA_FLAG_UNGATED_OUTPUT |
                              RLA_FLAG_DECAYED_RESIDUAL | RLA_FLAG_QK_SILU_L2NORM |
                              RLA_FLAG_GATE_PREACT;
  if (pp->flags & ~kKnown) return RLA_ERR_VALUE;
  pr.vflags = ((pp->flags & RLA_FLAG_RESIDUAL_TANH) ? kVarTanh : 0) |
              ((pp->flags & RLA_FLAG_UNGATED_OUTPUT) ? kVarUngated : 0) |
              ((pp->flags & RLA_FLAG_DECAYED_RESIDUAL) ? kVarDecayed : 0) |
              ((pp->flags & RLA_FLAG_GATE_PREACT) ? kVarGatePreact : 0) |
              ((pp->flags & RLA_FLAG_QK_SILU_L2NORM) ? kVarQkNorm : 0);
  if ((pp->flags & RLA_FLAG_GATE_PREACT) && !pp->decay_param) return RLA_ERR_NULL_ARG;
  pr.decay_param = pp->decay_param;
  pr.decay_param_grad = pp->decay_param_grad;
  pr.save = (pp->flags & RLA_FLAG_SAVE_FOR_BACKWARD) != 0;
  pr.use_saved = (pp->flags & RLA_FLAG_USE_SAVED) != 0;
  pr.B = pp->batch;
  pr.T = pp->seq_len;
  pr.H = pp->num_heads;
  pr.DK = pp->head_dim_k;
  pr.DV = pp->head_dim_v;
  pr.bf16 = pp->dtype == RLA_BF16;
  pr.out_bf16 = pp->out_dtype == RLA_BF16;
  pr.clip = isinf(pp->clip) ? -1.f : pp->clip;
  pr.cu = pp->cu_seqlens;
  pr.varlen = pp->cu_seqlens != nullptr;
  if (pr.varlen) {
    if (pr.B != 1 || pp->num_seqs < 0 || pp->num_seqs > (int64_t)1 << 30) return RLA_ERR_SHAPE;
    pr.N = pp->num_seqs;
    pr.ntok = pr.T;
    pr.max_chunks = pr.N == 0 ? 0 : (pr.T + kChunk - 1) / kChunk + pr.N;
  } else {
    pr.N = pr.B;
    if (pr.T > 0 && pr.B > INT64_MAX / pr.T) return RLA_ERR_SHAPE;
    pr.ntok = pr.B * pr.T;
    pr.max_chunks = pr.B * ((pr.T + kChunk - 1) / kChunk);
  }
  if (pr.max_chunks > INT32_MAX / 2 || pr.N * pr.H > INT32_MAX / 8) return RLA_ERR_SHAPE;
  return RLA_OK;
}

Workspace plan(const Problem& pr, int op) {
  Workspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t mc = (size_t)pr.max_chunks, H = (size_t)pr.H;
  if (pr.varlen) {
    w.seqs = take(sizeof(SeqInfo) * (size_t)pr.N);
    w.chunks = take(sizeof(ChunkInfo) * mc);
    w.nchunks = take(sizeof(int32_t));
    w.order = take(sizeof(int32_t) * (size_t)pr.N);
  }
  w.gates = take(sizeof(float) * mc * H * kGateBlock);
  const bool bwd = op == RLA_OP_RDN_BACKWARD || op == RLA_OP_RLA_BACKWARD;
  if (pr.vflags & kVarQkNorm) {   // normalised q, k (fp16 / fp32); backward: their fp32 gradients
    const size_t rows = (size_t)pr.ntok * H * (size_t)pr.DK;
    w.qh = take((pr.bf16 ? 2 : 4) * rows);
    w.kh = take((pr.bf16 ? 2 : 4) * rows);
    if (bwd) {
      w.dqh = take(4 * rows);
      w.dkh = take(4 * rows);
    }
  }
  if ((pr.vflags & kVarGatePreact) && bwd) w.dpart = take(sizeof(float) * mc * H * 2);
  w.mats = take((pr.bf16 ? 2 : 4) * mc * H * kNumMats * kMatElems);
  if (op == RLA_OP_RDN_BACKWARD || op == RLA_OP_RLA_BACKWARD) {
    // states: fp16 with per-(16 rows, 32 columns) scales for bf16 inputs, fp32 otherwise
    const size_t st = (pr.bf16 ? 2 : 4) * mc * H * (size_t)pr.DK * (size_t)pr.DV;
    const size_t sc = pr.bf16 ? sizeof(float) * mc * H * (size_t)(pr.DK / 16) * (size_t)(pr.DV / 32) : 0;
    w.ckS = take(st);
    w.ckR = take(st);
    w.mask = take((size_t)pr.ntok * H * (size_t)pr.DV);
    w.dS = take(st);
    w.dR = take(st);
    if (sc) {
      w.ckS_sc = take(sc);
      w.ckR_sc = take(sc);
      w.dS_sc = take(sc);
      w.dR_sc = take(sc);
    }
    const size_t bl = (pr.bf16 ? 2 : 4) * mc * H * kNumBlk * kChunk * (size_t)pr.DV;
    w.fblk = take(bl);
    w.bblk = take(bl);
    if (pr.bf16) {
      w.gmax = take(sizeof(uint32_t) * mc * H);
      w.gscale = take(sizeof(float) * (size_t)pr.N * H);
    }
  }
  w.total = off;
  return w;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

rla_status to_status(hipError_t e) { return e == hipSuccess ? RLA_OK : RLA_ERR_HIP; }

// Common set-up of OpParams from a validated problem and a workspace.
OpParams make_params(const Problem& pr, const Workspace& w, unsigned char* ws, bool rdn) {
  OpParams p;
  p.H = (int32_t)pr.H;
  p.DK = (int32_t)pr.DK;
  p.DV = (int32_t)pr.DV;
  p.ntok = pr.ntok;
  p.clip = pr.clip;
  p.rdn = rdn ? 1 : 0;
  p.vflags = pr.vflags;
  p.decay_param = pr.decay_param;
  p.out_bf16 = pr.out_bf16 ? 1 : 0;
  p.max_chunks = (int32_t)pr.max_chunks;
  p.st.nseq = (int32_t)pr.N;
  if (pr.varlen) {
    p.st.dense_T = -1;
    p.st.dense_nch = 0;
    p.st.seqs = reinterpret_cast<const SeqInfo*>(ws + w.seqs);
    p.st.chunks = reinterpret_cast<const ChunkInfo*>(ws + w.chunks);
    p.st.nchunks = reinterpret_cast<const int32_t*>(ws + w.nchunks);
    p.st.order = reinterpret_cast<const int32_t*>(ws + w.order);
  } else {
    p.st.dense_T = pr.T;
    p.st.dense_nch = (int32_t)((pr.T + kChunk - 1) / kChunk);
  }
  p.gate_ws = reinterpret_cast<float*>(ws + w.gates);
  p.mat_ws = ws + w.mats;
  return p;
}

// Workspace regions written by a saving forward and read by the backward.
void set_saved(const Problem& pr, const Workspace& w, unsigned char* ws, OpParams& p) {
  p.ck_S = ws + w.ckS;
  p.ck_R = ws + w.ckR;
  p.ck_mask = reinterpret_cast<uint8_t*>(ws + w.mask);
  p.dS_ws = ws + w.dS;
  p.dR_ws = ws + w.dR;
  if (pr.bf16) {
    p.ck_S_sc = reinterpret_cast<float*>(ws + w.ckS_sc);
    p.ck_R_sc = reinterpret_cast<float*>(ws + w.ckR_sc);
    p.dS_sc = reinterpret_cast<float*>(ws + w.dS_sc);
    p.dR_sc = reinterpret_cast<float*>(ws + w.dR_sc);
  }
  p.fwd_blk = ws + w.fblk;
  p.bwd_blk = ws + w.bblk;
}

rla_status check_workspace(const Workspace& w, void* ws, size_t bytes) {
  if (w.total == 0) return RLA_OK;
  if (!ws || bytes < w.total) return RLA_ERR_WORKSPACE;
  if (((uintptr_t)ws & (kAlign - 1)) != 0) return RLA_ERR_VALUE;
  return RLA_OK;
}

hipError_t build_tables(const Problem& pr, const Workspace& w, unsigned char* ws,
                        hipStream_t stream) {
  if (!pr.varlen || pr.N == 0) return hipSuccess;
  return launch_seq_table(pr.cu, (int32_t)pr.N, pr.ntok, (int32_t)pr.max_chunks,
                          reinterpret_cast<SeqInfo*>(ws + w.seqs),
                          reinterpret_cast<ChunkInfo*>(ws + w.chunks),
                          reinterpret_cast<int32_t*>(ws + w.nchunks),
                          reinterpret_cast<int32_t*>(ws + w.order), stream);
}

rla_status forward(bool rdn, const rla_problem* problem, const void* q, const void* k,
                   const void* v, const float* alpha_s, const float* beta, const float* alpha_r,
                   const float* gamma, const float* S0, const float* R0, void* o, float* S_final,
                   float* R_final, void* workspace, size_t workspace_bytes, void* stream_) {
  Problem pr;
  rla_status st = check_problem(problem, pr);
  if (st != RLA_OK) return st;
  if (pr.ntok > 0 && (!q || !k || !v || !alpha_s || !beta || !alpha_r || !gamma || !o))
    return RLA_ERR_NULL_ARG;
  if (pr.ntok > 0 && (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)))
    return RLA_ERR_VALUE;
  if (pr.save && !pr.bf16 && pr.DV != 64) return RLA_ERR_UNSUPPORTED;
  const int op = pr.save ? (rdn ? RLA_OP_RDN_BACKWARD : RLA_OP_RLA_BACKWARD)
                         : (rdn ? RLA_OP_RDN_FORWARD : RLA_OP_RLA_FORWARD);
  const Workspace w = plan(pr, op);
  st = check_workspace(w, workspace, workspace_bytes);
  if (st != RLA_OK) return st;
  if (pr.N == 0) return RLA_OK;

  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  unsigned char* ws = reinterpret_cast<unsigned char*>(workspace);
  OpParams p = make_params(pr, w, ws, rdn);
  p.q = q; p.k = k; p.v = v;
  p.alpha_s = alpha_s; p.beta = beta; p.alpha_r = alpha_r; p.gamma = gamma;
  p.S0 = S0; p.R0 = R0;
  p.o = o; p.S_fin = S_final; p.R_fin = R_final;
  if (pr.save) set_saved(pr, w, ws, p);

  hipError_t e = hipSuccess;
  if (pr.varlen && pr.ntok > 0)   // tokens outside every sequence read as zero
    e = launch_zero_fill(o, (size_t)pr.ntok * pr.H * pr.DV * (pr.out_bf16 ? 2 : 4), stream);
  if (e == hipSuccess) e = build_tables(pr, w, ws, stream);
  if (e == hipSuccess) e = mark_stage(stream, true);
  if (e == hipSuccess && (pr.vflags & kVarQkNorm)) {   // q, k -> SiLU + L2 norm rows
    e = launch_qk_norm_fwd(q, k, ws + w.qh, ws + w.kh, pr.ntok * pr.H, (int)pr.DK, pr.bf16, stream);
    p.q = ws + w.qh;
    p.k = ws + w.kh;
    p.qk_f16 = pr.bf16 ? 1 : 0;
  }
  if (e == hipSuccess) e = launch_prep(p, pr.bf16, stream);
  if (e == hipSuccess) e = mark_stage(stream, false);
  if (e == hipSuccess) e = launch_fwd_scan(p, pr.bf16, /*write_o=*/true, /*ckpt=*/pr.save, stream);
  if (e == hipSuccess) e = mark_stage(stream, false);
  return to_status(e);
}

rla_status backward(bool rdn, const rla_problem* problem, const void* q, const void* k, const void* v,
                        const float* alpha_s, const float* beta, const float* alpha_r,
                        const float* gamma, const float* S0, const float* R0, const void* dO,
                        const float* dS_final, const float* dR_final, void* dq, void* dk,
                        void* dv, float* dalpha_s, float* dbeta, float* dalpha_r, float* dgamma,
                        float* dS0, float* dR0, void* workspace, size_t workspace_bytes,
                        void* stream_) {
  Problem pr;
  rla_status st = check_problem(problem, pr);
  if (st != RLA_OK) return st;
  if (pr.ntok > 0 && (!q || !k || !v || !alpha_s || !beta || !alpha_r || !gamma || !dO ||
                      !dq || !dk || !dv || !dalpha_s || !dbeta || !dalpha_r || !dgamma))
    return RLA_ERR_NULL_ARG;
  if (pr.ntok > 0 && (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dO) ||
                      !aligned16(dq) || !aligned16(dk) || !aligned16(dv)))
    return RLA_ERR_VALUE;
  if (!pr.bf16 && pr.DV != 64) return RLA_ERR_UNSUPPORTED;
  const Workspace w = plan(pr, rdn ? RLA_OP_RDN_BACKWARD : RLA_OP_RLA_BACKWARD);
  st = check_workspace(w, workspace, workspace_bytes);
  if (st != RLA_OK) return st;
  if (pr.N == 0) return RLA_OK;

  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  unsigned char* ws = reinterpret_cast<unsigned char*>(workspace);
  OpParams p = make_params(pr, w, ws, rdn);
  p.q = q; p.k = k; p.v = v;
  p.alpha_s = alpha_s; p.beta = beta; p.alpha_r = alpha_r; p.gamma = gamma;
  p.S0 = S0; p.R0 = R0;
  set_saved(pr, w, ws, p);
  p.dO = dO; p.dS_fin = dS_final; p.dR_fin = dR_final;
  p.dq = dq; p.dk = dk; p.dv = dv;
  p.dalpha_s = dalpha_s; p.dbeta = dbeta; p.dalpha_r = dalpha_r; p.dgamma = dgamma;
  p.dS0 = dS0; p.dR0 = dR0;

  hipError_t e = hipSuccess;
  if (pr.varlen && pr.ntok > 0) {   // tokens outside every sequence get zero gradients
    const size_t el = pr.out_bf16 ? 2 : 4, tok = (size_t)pr.ntok * pr.H;
    e = launch_zero_fill(dq, tok * pr.DK * el, stream);
    if (e == hipSuccess) e = launch_zero_fill(dk, tok * pr.DK * el, stream);
    if (e == hipSuccess) e = launch_zero_fill(dv, tok * pr.DV * el, stream);
    if (e == hipSuccess) e = launch_zero_fill(dalpha_s, tok * 4, stream);
    if (e == hipSuccess) e = launch_zero_fill(dbeta, tok * 4, stream);
    if (e == hipSuccess) e = launch_zero_fill(dalpha_r, tok * 4, stream);
    if (e == hipSuccess) e = launch_zero_fill(dgamma, tok * 4, stream);
  }
  if (e == hipSuccess && !pr.use_saved) e = build_tables(pr, w, ws, stream);
  if (e == hipSuccess) e = mark_stage(stream, true);
  const bool qkn = (pr.vflags & kVarQkNorm) != 0;
  if (qkn) {   // the chunked path reads the normalised rows (saved by a saving forward)
    if (e == hipSuccess && !pr.use_saved)
      e = launch_qk_norm_fwd(q, k, ws + w.qh, ws + w.kh, pr.ntok * pr.H, (int)pr.DK, pr.bf16, stream);
    p.q = ws + w.qh;
    p.k = ws + w.kh;
    p.qk_f16 = pr.bf16 ? 1 : 0;
    // the gradient kernel writes d(normalised q, k) in fp32 into the workspace
    p.dq = ws + w.dqh;
    p.dk = ws + w.dkh;
    if (e == hipSuccess && pr.varlen) {   // rows outside every sequence stay zero
      const size_t bytes = (size_t)pr.ntok * pr.H * pr.DK * 4;
      e = launch_zero_fill(ws + w.dqh, bytes, stream);
      if (e == hipSuccess) e = launch_zero_fill(ws + w.dkh, bytes, stream);
    }
  }
  const bool pre = (pr.vflags & kVarGatePreact) != 0;
  if (pre) {
    p.decay_partials = reinterpret_cast<float*>(ws + w.dpart);
    if (e == hipSuccess)
      e = launch_zero_fill(ws + w.dpart, sizeof(float) * (size_t)pr.max_chunks * pr.H * 2, stream);
  }
  if (!pr.use_saved) {
    if (e == hipSuccess) e = launch_prep(p, pr.bf16, stream);
    if (e == hipSuccess) e = mark_stage(stream, false);
    if (e == hipSuccess) e = launch_fwd_scan(p, pr.bf16, /*write_o=*/false, /*ckpt=*/true, stream);
    if (e == hipSuccess) e = mark_stage(stream, false);
  }
  if (pr.bf16) {   // one power-of-two scale of the upstream gradients per (sequence, head)
    p.grad_absmax = reinterpret_cast<const uint32_t*>(ws + w.gmax);
    p.grad_scale = reinterpret_cast<float*>(ws + w.gscale);
    if (e == hipSuccess) e = launch_grad_absmax(p, reinterpret_cast<uint32_t*>(ws + w.gmax), stream);
    if (e == hipSuccess) e = mark_stage(stream, false);
  }
  if (e == hipSuccess) e = launch_bwd_scan(p, pr.bf16, stream);
  if (e == hipSuccess) e = mark_stage(stream, false);
  {
    OpParams pg = p;
    if (qkn) pg.out_bf16 = 0;   // fp32 gradients of the normalised rows
    if (e == hipSuccess) e = launch_bwd_grad(pg, pr.bf16, stream);
  }
  if (e == hipSuccess && qkn)
    e = launch_qk_norm_bwd(q, k, reinterpret_cast<const float*>(ws + w.dqh),
                           reinterpret_cast<const float*>(ws + w.dkh), dq, dk, pr.ntok * pr.H,
                           (int)pr.DK, pr.bf16, pr.out_bf16, stream);
  if (e == hipSuccess && pre && pr.decay_param_grad)
    e = launch_decay_grad_reduce(p.decay_partials, (int)pr.max_chunks, (int)pr.H,
                                 pr.decay_param_grad, stream);
  if (e == hipSuccess) e = mark_stage(stream, false);
  return to_status(e);
}


// Byte ranges [a, a + bytes) and [b, b + bytes) intersect (NULL never does).
bool ranges_overlap(const void* a, const void* b, size_t bytes) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  if (!a || !b) return false;
  return x < y + bytes && y < x + bytes;
}

rla_status decode(bool rdn, const rla_problem* problem, const void* q, const void* k,
                  const void* v, const float* alpha_s, const float* beta, const float* alpha_r,
                  const float* gamma, const float* S_in, const float* R_in, void* o,
                  float* S_out, float* R_out, void* stream_) {
  Problem pr;
  rla_status st = check_problem(problem, pr, /*recurrent=*/true);
  if (st != RLA_OK) return st;
  if (pr.varlen) return RLA_ERR_UNSUPPORTED;
  if (pr.save || pr.use_saved) return RLA_ERR_VALUE;
  if (pr.N * pr.H == 0) return RLA_OK;
  if (!S_out || !R_out) return RLA_ERR_NULL_ARG;
  if (pr.ntok > 0 && (!q || !k || !v || !alpha_s || !beta || !alpha_r || !gamma || !o))
    return RLA_ERR_NULL_ARG;
  if (pr.ntok > 0 && (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)))
    return RLA_ERR_VALUE;
  if ((S_in && !aligned16(S_in)) || (R_in && !aligned16(R_in)) || !aligned16(S_out) ||
      !aligned16(R_out))
    return RLA_ERR_VALUE;
  const size_t sbytes = (size_t)pr.N * pr.H * pr.DK * pr.DV * sizeof(float);
  // outputs may alias their own input exactly (in-place), nothing else
  if ((S_in != S_out && ranges_overlap(S_in, S_out, sbytes)) ||
      (R_in != R_out && ranges_overlap(R_in, R_out, sbytes)) ||
      ranges_overlap(S_out, R_out, sbytes) || ranges_overlap(S_in, R_out, sbytes) ||
      ranges_overlap(R_in, S_out, sbytes))
    return RLA_ERR_VALUE;
  if ((int64_t)pr.N * pr.H > INT32_MAX / 4 || pr.T > INT32_MAX) return RLA_ERR_SHAPE;

  OpParams p;
  p.H = (int32_t)pr.H;
  p.DK = (int32_t)pr.DK;
  p.DV = (int32_t)pr.DV;
  p.ntok = pr.ntok;
  p.clip = pr.clip;
  p.rdn = rdn ? 1 : 0;
  p.vflags = pr.vflags;
  p.decay_param = pr.decay_param;
  p.out_bf16 = pr.out_bf16 ? 1 : 0;
  p.st.nseq = (int32_t)pr.N;
  p.st.dense_T = pr.T;
  p.q = q; p.k = k; p.v = v;
  p.alpha_s = alpha_s; p.beta = beta; p.alpha_r = alpha_r; p.gamma = gamma;
  p.S0 = S_in; p.R0 = R_in;
  p.o = o; p.S_fin = S_out; p.R_fin = R_out;
  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  hipError_t e = mark_stage(stream, true);
  if (e == hipSuccess) e = launch_decode(p, pr.bf16, stream);
  if (e == hipSuccess) e = mark_stage(stream, false);
  return to_status(e);
}

// ---- allocation-free forward: the workspace is a static device array ----
// Each GPU the library runs on holds its own copy from the first use until the
// process ends.  Host code must not use the array's name as a device address:
// the address is taken once per device with hipGetSymbolAddress (with that
// device current) and kept in scratch_ptr.
constexpr size_t kScratchBytes = size_t(RLA_NOALLOC_SCRATCH_BYTES);
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 256;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (taken on its first use).
rla_status current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RLA_ERR_HIP;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return RLA_ERR_HIP;
    scratch_ptr[dev] = ptr;
  }
  *out = scratch_ptr[dev];
  return RLA_OK;
}

}  // namespace
}  // namespace rla

using namespace rla;

extern "C" {

size_t rla_workspace_size(const rla_problem* problem, int op) {
  Problem pr;
  if (check_problem(problem, pr) != RLA_OK) return 0;
  if (op < RLA_OP_RLA_FORWARD || op > RLA_OP_RLA_BACKWARD) return 0;
  return plan(pr, op).total;
}

void rla_set_stage_events(void** events, int num_events) {
  g_events = reinterpret_cast<hipEvent_t*>(events);
  g_num_events = events ? num_events : 0;
  g_next_event = 0;
}

const char* rla_status_string(rla_status s) {
  switch (s) {
    case RLA_OK: return "ok";
    case RLA_ERR_NULL_ARG: return "required pointer is NULL";
    case RLA_ERR_SHAPE: return "unsupported or inconsistent shape";
    case RLA_ERR_DTYPE: return "unsupported dtype for this shape";
    case RLA_ERR_UNSUPPORTED: return "not implemented";
    case RLA_ERR_WORKSPACE: return "workspace missing or too small";
    case RLA_ERR_VALUE: return "bad scalar argument or misaligned pointer";
    case RLA_ERR_HIP: return "HIP runtime error";
    case RLA_ERR_SCRATCH: return "problem needs more workspace than the static scratch holds";
  }
  return "unknown status";
}

rla_status rla_forward(const rla_problem* problem, const void* q, const void* k, const void* v,
                       const float* alpha_s, const float* beta, const float* alpha_r,
                       const float* gamma, const float* S0, const float* R0, void* o,
                       float* S_final, float* R_final, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return forward(false, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S0, R0, o, S_final,
                 R_final, workspace, workspace_bytes, stream);
}

rla_status rdn_forward(const rla_problem* problem, const void* q, const void* k, const void* v,
                       const float* alpha_s, const float* beta, const float* alpha_r,
                       const float* gamma, const float* S0, const float* R0, void* o,
                       float* S_final, float* R_final, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return forward(true, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S0, R0, o, S_final,
                 R_final, workspace, workspace_bytes, stream);
}

rla_status rdn_forward_noalloc(const rla_problem* problem, const void* q, const void* k,
                               const void* v, const float* alpha_s, const float* beta,
                               const float* alpha_r, const float* gamma, const float* S0,
                               const float* R0, void* o, float* S_final, float* R_final,
                               void* stream) {
  Problem pr;
  rla_status st = check_problem(problem, pr);
  if (st != RLA_OK) return st;
  if (pr.save || pr.use_saved) return RLA_ERR_VALUE;
  if (plan(pr, RLA_OP_RDN_FORWARD).total > kScratchBytes) return RLA_ERR_SCRATCH;
  void* ws = nullptr;
  if (pr.N > 0) {
    st = current_scratch(&ws);
    if (st != RLA_OK) return st;
  }
  return forward(true, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S0, R0, o, S_final,
                 R_final, ws, kScratchBytes, stream);
}

rla_status rla_backward(const rla_problem* problem, const void* q, const void* k, const void* v,
                        const float* alpha_s, const float* beta, const float* alpha_r,
                        const float* gamma, const float* S0, const float* R0, const void* dO,
                        const float* dS_final, const float* dR_final, void* dq, void* dk,
                        void* dv, float* dalpha_s, float* dbeta, float* dalpha_r, float* dgamma,
                        float* dS0, float* dR0, void* workspace, size_t workspace_bytes,
                        void* stream) {
  return backward(false, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S0, R0, dO, dS_final,
                  dR_final, dq, dk, dv, dalpha_s, dbeta, dalpha_r, dgamma, dS0, dR0, workspace,
                  workspace_bytes, stream);
}

rla_status rdn_backward(const rla_problem* problem, const void* q, const void* k, const void* v,
                        const float* alpha_s, const float* beta, const float* alpha_r,
                        const float* gamma, const float* S0, const float* R0, const void* dO,
                        const float* dS_final, const float* dR_final, void* dq, void* dk,
                        void* dv, float* dalpha_s, float* dbeta, float* dalpha_r, float* dgamma,
                        float* dS0, float* dR0, void* workspace, size_t workspace_bytes,
                        void* stream) {
  return backward(true, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S0, R0, dO, dS_final,
                  dR_final, dq, dk, dv, dalpha_s, dbeta, dalpha_r, dgamma, dS0, dR0, workspace,
                  workspace_bytes, stream);
}

rla_status rla_decode(const rla_problem* problem, const void* q, const void* k, const void* v,
                      const float* alpha_s, const float* beta, const float* alpha_r,
                      const float* gamma, const float* S_in, const float* R_in, void* o,
                      float* S_out, float* R_out, void* stream) {
  return decode(false, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S_in, R_in, o, S_out,
                R_out, stream);
}

rla_status rdn_decode(const rla_problem* problem, const void* q, const void* k, const void* v,
                      const float* alpha_s, const float* beta, const float* alpha_r,
                      const float* gamma, const float* S_in, const float* R_in, void* o,
                      float* S_out, float* R_out, void* stream) {
  return decode(true, problem, q, k, v, alpha_s, beta, alpha_r, gamma, S_in, R_in, o, S_out,
                R_out, stream);
}

}  // extern "C"
