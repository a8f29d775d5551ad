// luna_api.cpp -- host side of the C ABI declared in include/luna.h.
//
// Every entry point validates its arguments completely on the host before any HIP
// call, plans the workspace (piecewise-linear tables first, then per-operation
// buffers, each 256-byte aligned) and enqueues its kernels on the caller's stream.
#include "luna.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <mutex>
#include <string>

#include "luna_kernels.hpp"

namespace {

thread_local std::string g_last_error;

luna_status fail(luna_status s, const std::string& why) {
  g_last_error = why;
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Problem {
  int op;
  luna_dtype dt;
  int64_t B, H, n, d;
  const luna_phi_params* p;
  int32_t chunk;
};

int param_sets(const Problem& pb) { return pb.p->per_head ? (int)pb.H : 1; }

// Checks shared by every operation; `why` receives the reason on failure.
luna_status check_common(const Problem& pb) {
  const luna_phi_params* p = pb.p;
  if (p == nullptr) return fail(LUNA_ERR_INVALID_ARG, "params is NULL");
  if (pb.dt != LUNA_F32 && pb.dt != LUNA_BF16) return fail(LUNA_ERR_INVALID_ARG, "dtype must be LUNA_F32 or LUNA_BF16");
  if (pb.B < 1 || pb.H < 1 || pb.n < 1) return fail(LUNA_ERR_INVALID_ARG, "B, H and n must be >= 1");
  if (pb.n > (int64_t)1 << 30) return fail(LUNA_ERR_UNSUPPORTED, "n must be <= 2^30");
  if (pb.B * pb.H > (int64_t)1 << 24) return fail(LUNA_ERR_UNSUPPORTED, "B*H must be <= 2^24");
  if (pb.d != 32 && pb.d != 64 && pb.d != 128) return fail(LUNA_ERR_UNSUPPORTED, "d must be 32, 64 or 128");
  if (p->M < 1 || p->M > 256) return fail(LUNA_ERR_INVALID_ARG, "M must be in [1, 256]");
  if (p->L < 1 || p->L > 16) return fail(LUNA_ERR_INVALID_ARG, "L must be in [1, 16]");
  if (p->hidden < 1 || p->hidden > 64) return fail(LUNA_ERR_INVALID_ARG, "hidden must be in [1, 64]");
  if (p->M * p->L > 256) return fail(LUNA_ERR_INVALID_ARG, "M*L must be <= 256");
  if (p->shared_channels != 0 && p->shared_channels != 1) return fail(LUNA_ERR_INVALID_ARG, "shared_channels must be 0 or 1");
  if (p->nonneg != 0 && p->nonneg != 1) return fail(LUNA_ERR_INVALID_ARG, "nonneg must be 0 or 1");
  if (p->per_head != 0 && p->per_head != 1) return fail(LUNA_ERR_INVALID_ARG, "per_head must be 0 or 1");
  if (!p->W || !p->b || !p->fc1_w || !p->fc1_b || !p->fc2_w || !p->fc2_b)
    return fail(LUNA_ERR_INVALID_ARG, "a parameter array is NULL");
  const int C1 = p->shared_channels ? 1 : p->L;
  const int units = C1 * p->hidden;
  if (units > luna::kMaxUnits) return fail(LUNA_ERR_UNSUPPORTED, "L*hidden must be <= 1023 (breakpoint table)");
  // the feature-map kernel (also the first stage of a streaming step) has the larger LDS table
  const bool fm_table = pb.op == LUNA_OP_FEATUREMAP || pb.op == LUNA_OP_CAUSAL_STEP || pb.op == LUNA_OP_ATTN_BWD ||
                        pb.op == LUNA_OP_ATTN_CAUSAL_BWD || pb.op >= 100;
  const int seg_cap = luna::nseg_cap(p->L, fm_table ? luna::kFmSegBytes : luna::kAttnSegBytes);
  if (units + 2 > seg_cap) return fail(LUNA_ERR_UNSUPPORTED, "too many breakpoints for the LDS segment table");
  if ((units + 1) * p->L > luna::kSegCap || (size_t)(units + 1) * luna::seg16_row_bytes(p->L) > luna::kSeg16Bytes)
    return fail(LUNA_ERR_UNSUPPORTED, "too many segments for the table");
  return LUNA_OK;
}

struct Layout {
  size_t tables = 0, partial = 0, frags = 0, total = 0;
  size_t phiq = 0, phik = 0;  // streaming step: features of the new queries and keys (fp32)
  size_t zcopy = 0;           // streaming step: z as it was before the call
  // backward pass: [V | 1], [num | den] then [dnum | dden], per-chunk states and their
  // gradients, intra-chunk P and R (causal), feature gradients, dV in fp32 (bf16
  // calls), per-workgroup parameter partials, their fp64 sums and moment prefixes
  size_t vx = 0, y = 0, sx = 0, dsx = 0, pm = 0, rm = 0, dphiq = 0, dphik = 0, dvtmp = 0;
  size_t xq = 0, xk = 0, wx = 0, uq = 0, uk = 0, duq = 0, duk = 0, dwh = 0;  // feature-map backward
  size_t bpart = 0, sum = 0, pre = 0;
  size_t dstats = 0;  // distillation: per query row the softmax max and sum and the kernel row sum
  int chunk = 0, nch = 1, groups = 0, part_floats = 0;
  int splits = 1, tokens_per_split = 0, tile_tokens = 256, tiles = 1, fused = 0;
  int parts = 1, split = 0;  // causal: workgroups per head, first token of part 1
  size_t state = 0;          // causal with 2 parts: state pieces of the first `split` tokens
  int pieces = 0, piece_chunks = 0;
  int staged = 0, sa = 0, sb = 0;  // staged causal scan: chunks of the first scanned part and of the state-only part
  int generic = 0;  // forward in fp32 GEMMs and scans (shapes without a fused kernel)
  int given = 0;    // causal: features mapped beforehand (bf16, in phiq / phik), then the scan kernel
};

// Buffers of the forward pass in fp32 GEMMs (the forward of shapes without a fused
// kernel, and the recomputation that starts the backward pass): features of the keys
// (and queries), [V | 1], [num | den - eps] and the per-chunk states, plus P for the
// causal form.  Causal chunks are the 64-token chunks of the scan; the non-causal form
// cuts its sums over tokens into 512-token pieces, for parallelism only.
// (features: the buffers for fp32 features, or none when the caller's are used)
luna_status plan_f32_buffers(int64_t heads, int64_t n, int d, int D, bool causal, bool queries, bool features,
                             Layout* lay, size_t* off) {
  lay->chunk = causal ? 64 : 512;
  const int64_t nch = (n + lay->chunk - 1) / lay->chunk;
  if (nch > 65535) return fail(LUNA_ERR_UNSUPPORTED, causal ? "n must be <= 65535 * 64" : "n must be <= 65535 * 512");
  lay->nch = (int)nch;
  const size_t rows = (size_t)heads * (size_t)n, states = (size_t)heads * lay->nch;
  auto take = [&](size_t& at, size_t bytes) {
    at = *off;
    *off = align256(*off + bytes);
  };
  if (queries && features) take(lay->phiq, rows * D * 4);
  if (features) take(lay->phik, rows * D * 4);
  take(lay->vx, rows * (d + 1) * 4);
  if (queries) take(lay->y, rows * (d + 1) * 4);
  take(lay->sx, states * D * (d + 1) * 4);
  if (causal && queries) take(lay->pm, states * 64 * 64 * 4);
  return LUNA_OK;
}
luna_status plan_f32_forward(const Problem& pb, bool causal, bool queries, Layout* lay, size_t* off) {
  return plan_f32_buffers(pb.B * pb.H, pb.n, (int)pb.d, pb.p->M * pb.p->L, causal, queries, true, lay, off);
}

// The causal kernel's split.  Too few heads to fill the device: with 97 to 128 heads
// the staged form below (two scan launches); otherwise cut every head in two at a
// chunk boundary x near n/2, where a state launch first sums the state of [0, x) in
// pieces (one workgroup per head and piece, enough pieces to fill the device) and part
// 1 of the scan launch starts from the sum of the pieces.
void plan_causal_parts(int64_t heads, int64_t n, size_t state_floats, Layout* lay, size_t* off, bool staged_ok) {
  const int64_t nch = (n + 63) / 64;
  if (staged_ok && heads > 96 && heads <= 128 && nch >= 5) {
    // Two workgroups per head fill the device, so both launches are scan launches
    // (staged): the first scans chunks [0, A) of every head and, beside it, sums the
    // state of [A, A + B); the second scans [A, A + B) and [A + B, nch) from those
    // states.  A state-only chunk costs about half a scanned one, so A = nch / 5 and
    // B = C = 2 nch / 5 balance both launches (about 153 scanned-chunk times for 256
    // chunks, against 161 for a state launch over [0, nch / 2) followed by two
    // scanned halves).
    const int64_t A = (nch + 2) / 5;
    const int64_t B = (nch - A) / 2;
    lay->parts = 2;
    lay->staged = 1;
    lay->sa = (int)A;
    lay->sb = (int)B;
    lay->split = (int)(64 * A);
    lay->pieces = 2;
    lay->piece_chunks = 0;
    lay->state = *off;
    *off = align256(*off + (size_t)heads * 2 * state_floats * sizeof(float));
    return;
  }
  if (heads < 256 && n >= 256) {
    const int64_t cx = n / 64 / 2;  // chunks before the split
    if (cx >= 1) {
      lay->parts = 2;
      lay->split = (int)(cx * 64);
      int64_t pieces = (256 + heads - 1) / heads;
      if (pieces > cx) pieces = cx;
      const int64_t pc = (cx + pieces - 1) / pieces;
      lay->piece_chunks = (int)pc;
      lay->pieces = (int)((cx + pc - 1) / pc);  // every piece non-empty
      lay->state = *off;
      *off = align256(*off + (size_t)heads * lay->pieces * state_floats * sizeof(float));
    }
  }
}

// Token ranges of the non-causal state pass: enough state workgroups to fill the
// device, at least 256 tokens each, a multiple of 128 tokens per range.
void plan_splits(const Problem& pb, int64_t heads, Layout* lay) {
  const int64_t want = (512 + heads - 1) / heads;
  const int64_t maxs = (pb.n + 255) / 256;
  int64_t splits = want < maxs ? want : maxs;
  if (splits < 1) splits = 1;
  int64_t tps = (pb.n + splits - 1) / splits;
  tps = (tps + 127) / 128 * 128;
  splits = (pb.n + tps - 1) / tps;
  lay->splits = (int)splits;
  lay->tokens_per_split = (int)tps;
}

// Private operation codes of the distillation loss (without and with the feature-map
// parameter gradients).
constexpr int kOpDistill = 100, kOpDistillGrads = 101;

// Buffers of the feature-map backward (enqueue_phi_backward): [x | 1] of the queries
// and keys, [W | b], the projections and their gradients, per-(batch, head) [dW | db],
// the per-workgroup parameter partials, their fp64 sums and moment prefixes.
void plan_phi_backward(const Problem& pb, Layout* lay, size_t* off) {
  const int d = (int)pb.d, L = pb.p->L, M = pb.p->M, P = param_sets(pb);
  const int64_t heads = pb.B * pb.H;
  const size_t rows = (size_t)heads * (size_t)pb.n;
  auto take = [&](size_t& at, size_t bytes) {
    at = *off;
    *off = align256(*off + bytes);
  };
  take(lay->xq, rows * (d + 1) * 4);
  take(lay->xk, rows * (d + 1) * 4);
  take(lay->wx, (size_t)P * M * (d + 1) * 4);
  take(lay->uq, rows * M * 4);
  take(lay->uk, rows * M * 4);
  take(lay->duq, rows * M * 4);
  take(lay->duk, rows * M * 4);
  take(lay->dwh, (size_t)heads * M * (d + 1) * 4);
  lay->groups = luna::bwd_phi_groups(2 * pb.n * (heads / P) * M);
  lay->part_floats = (int)luna::bwd_part_floats(d, L, M);
  take(lay->bpart, (size_t)P * lay->groups * lay->part_floats * 4);
  take(lay->sum, (size_t)P * lay->part_floats * 8);
  take(lay->pre, (size_t)P * L * (luna::bwd_nseg_cap(L) + 1) * 2 * 8);
}

luna_status plan(const Problem& pb, Layout* lay) {
  luna_status st = check_common(pb);
  if (st != LUNA_OK) return st;
  const luna::Dt dt = pb.dt == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int d = (int)pb.d, L = pb.p->L, M = pb.p->M;
  const int64_t heads = pb.B * pb.H;
  size_t off = 0;
  lay->tables = off;
  off = align256(off + (size_t)param_sets(pb) * luna::kTableBytes);
  if (pb.op == LUNA_OP_FEATUREMAP) {
    if (!luna::featuremap_supported(dt, d, L, M))
      return fail(LUNA_ERR_UNSUPPORTED, "no feature-map kernel for this (d, L, M)");
  } else if (pb.op == LUNA_OP_ATTN) {
    luna::NoncausalPlan np;
    if (!luna::noncausal_supported(dt, d, L, M, &np)) {
      if (!luna::featuremap_supported(dt, d, L, M))
        return fail(LUNA_ERR_UNSUPPORTED, "no non-causal attention kernels for this (dtype, d, L, M)");
      lay->generic = 1;
      if ((st = plan_f32_forward(pb, false, true, lay, &off)) != LUNA_OK) return st;
      lay->total = off;
      return LUNA_OK;
    }
    if (heads >= luna::kFusedMinHeads && luna::fused_acc_regs(d, L, M) <= luna::kFusedMaxAccRegs) {
      lay->fused = 1;
      lay->total = off;
      return LUNA_OK;
    }
    plan_splits(pb, heads, lay);
    lay->tile_tokens = 256;
    lay->tiles = (int)((pb.n + 255) / 256);
    lay->partial = off;
    off = align256(off + (size_t)heads * lay->splits * np.DP * (d + 1) * sizeof(float));
    lay->frags = off;
    off = align256(off + (size_t)heads * np.frag_elems * (pb.dt == LUNA_BF16 ? 2 : 4));
  } else if (pb.op == LUNA_OP_ATTN_CAUSAL) {
    if (pb.chunk != 64) return fail(LUNA_ERR_UNSUPPORTED, "chunk must be 64");
    size_t state_floats = 0;
    if (luna::causal_supported(dt, d, L, M)) {
      state_floats = luna::causal_state_floats(dt, d, L, M);
    } else if (!luna::featuremap_supported(dt, d, L, M)) {
      return fail(LUNA_ERR_UNSUPPORTED, "no causal attention kernels for this (dtype, d, L, M)");
    } else if (luna::causal_given_supported(dt, d, M * L)) {
      // the features of Q and K in bf16, mapped by the feature-map kernel
      lay->given = 1;
      state_floats = luna::causal_given_state_floats(d, M * L);
      const size_t feat_bytes = (size_t)heads * (size_t)pb.n * (size_t)(M * L) * 2;
      lay->phiq = off;
      off = align256(off + feat_bytes);
      lay->phik = off;
      off = align256(off + feat_bytes);
    } else {
      lay->generic = 1;
      if ((st = plan_f32_forward(pb, true, true, lay, &off)) != LUNA_OK) return st;
      lay->total = off;
      return LUNA_OK;
    }
    plan_causal_parts(heads, pb.n, state_floats, lay, &off, !lay->given);
  } else if (pb.op == LUNA_OP_STATE) {
    luna::NoncausalPlan np;
    if (luna::noncausal_supported(dt, d, L, M, &np)) {
      // the state pass of the non-causal split path
      plan_splits(pb, heads, lay);
      lay->partial = off;
      off = align256(off + (size_t)heads * lay->splits * np.DP * (d + 1) * sizeof(float));
    } else if (luna::causal_supported(dt, d, L, M)) {
      // the causal kernel's state launch over every chunk, in pieces
      const int64_t cx = (pb.n + 63) / 64;
      int64_t pieces = (256 + heads - 1) / heads;
      if (pieces > cx) pieces = cx;
      const int64_t pc = (cx + pieces - 1) / pieces;
      lay->piece_chunks = (int)pc;
      lay->pieces = (int)((cx + pc - 1) / pc);
      lay->split = (int)(cx * 64);
      lay->state = off;
      off = align256(off + (size_t)heads * lay->pieces * luna::causal_state_floats(dt, d, L, M) * sizeof(float));
    } else if (luna::featuremap_supported(dt, d, L, M)) {
      lay->generic = 1;
      if ((st = plan_f32_forward(pb, false, false, lay, &off)) != LUNA_OK) return st;
    } else {
      return fail(LUNA_ERR_UNSUPPORTED, "no state kernels for this (dtype, d, L, M)");
    }
  } else if (pb.op == LUNA_OP_CAUSAL_STEP) {
    if (!luna::featuremap_supported(dt, d, L, M))
      return fail(LUNA_ERR_UNSUPPORTED, "no feature-map kernel for this (d, L, M)");
    const size_t feat_bytes = (size_t)heads * (size_t)pb.n * (size_t)(M * L) * sizeof(float);
    lay->phiq = off;
    off = align256(off + feat_bytes);
    lay->phik = off;
    off = align256(off + feat_bytes);
    lay->zcopy = off;
    off = align256(off + (size_t)heads * (size_t)(M * L) * sizeof(float));
  } else if (pb.op == LUNA_OP_ATTN_BWD || pb.op == LUNA_OP_ATTN_CAUSAL_BWD) {
    if (!luna::bwd_supported(d, L, M) || !luna::featuremap_supported(dt, d, L, M))
      return fail(LUNA_ERR_UNSUPPORTED, "no backward kernels for this (d, L, M)");
    const int64_t P = param_sets(pb);
    if (P > 65535) return fail(LUNA_ERR_UNSUPPORTED, "at most 65535 parameter sets in the backward pass");
    if (pb.H > 65535) return fail(LUNA_ERR_UNSUPPORTED, "at most 65535 heads in the backward pass");
    const bool causal = pb.op == LUNA_OP_ATTN_CAUSAL_BWD;
    if ((st = plan_f32_forward(pb, causal, true, lay, &off)) != LUNA_OK) return st;
    const size_t D = (size_t)M * L, rows = (size_t)heads * (size_t)pb.n, states = (size_t)heads * lay->nch;
    auto take = [&](size_t& at, size_t bytes) {
      at = off;
      off = align256(off + bytes);
    };
    take(lay->dsx, states * D * (d + 1) * 4);
    if (causal) take(lay->rm, states * 64 * 64 * 4);
    take(lay->dphiq, rows * D * 4);
    take(lay->dphik, rows * D * 4);
    if (pb.dt == LUNA_BF16) take(lay->dvtmp, rows * d * 4);
    plan_phi_backward(pb, lay, &off);
  } else if (pb.op == kOpDistill || pb.op == kOpDistillGrads) {
    const int D = M * L;
    if (!luna::distill_supported(dt, d, D) || !luna::featuremap_supported(dt, d, L, M))
      return fail(LUNA_ERR_UNSUPPORTED, "no distillation kernels for this (dtype, d, M*L)");
    const size_t rows = (size_t)heads * (size_t)pb.n;
    auto take = [&](size_t& at, size_t bytes) {
      at = off;
      off = align256(off + bytes);
    };
    take(lay->phiq, rows * D * (pb.dt == LUNA_BF16 ? 2 : 4));  // features in the call's dtype
    take(lay->phik, rows * D * (pb.dt == LUNA_BF16 ? 2 : 4));
    take(lay->dstats, rows * 4 * sizeof(float));
    if (pb.op == kOpDistillGrads) {
      if (!luna::bwd_supported(d, L, M)) return fail(LUNA_ERR_UNSUPPORTED, "no backward kernels for this (d, L, M)");
      if (param_sets(pb) > 65535 || pb.H > 65535)
        return fail(LUNA_ERR_UNSUPPORTED, "at most 65535 heads and parameter sets in the backward pass");
      take(lay->dphiq, rows * D * 4);
      take(lay->dphik, rows * D * 4);
      plan_phi_backward(pb, lay, &off);
    }
  } else {
    return fail(LUNA_ERR_INVALID_ARG, "unknown operation code");
  }
  lay->total = off;
  return LUNA_OK;
}

luna_status check_ws(const Layout& lay, void* ws, size_t ws_bytes) {
  if (ws_bytes < lay.total) {
    char buf[128];
    snprintf(buf, sizeof buf, "workspace too small: need %zu bytes, got %zu", lay.total, ws_bytes);
    return fail(LUNA_ERR_WORKSPACE, buf);
  }
  if (ws == nullptr) return fail(LUNA_ERR_INVALID_ARG, "workspace is NULL");
  if (((uintptr_t)ws & 255) != 0) return fail(LUNA_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  return LUNA_OK;
}

luna_status hip_fail(hipError_t e, const char* what) {
  return fail(LUNA_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

luna_status enqueue_prepare(const Problem& pb, uint8_t* ws, const Layout& lay, hipStream_t s) {
  const luna_phi_params* p = pb.p;
  luna::PrepareArgs a{};
  a.fc1_w = p->fc1_w;
  a.fc1_b = p->fc1_b;
  a.fc2_w = p->fc2_w;
  a.fc2_b = p->fc2_b;
  a.P = param_sets(pb);
  a.C1 = p->shared_channels ? 1 : p->L;
  a.L = p->L;
  a.hidden = p->hidden;
  a.M = p->M;
  a.nonneg = p->nonneg;
  a.tables = ws + lay.tables;
  hipError_t e = luna::launch_prepare(a, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "table kernel launch");
}

luna::PhiArgs phi_args(const Problem& pb, uint8_t* ws, const Layout& lay) {
  luna::PhiArgs f{};
  f.W = pb.p->W;
  f.b = pb.p->b;
  f.tables = ws + lay.tables;
  f.M = pb.p->M;
  f.per_head = pb.p->per_head;
  return f;
}

bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.0f; }

// C (+)= A B (fp32) over (head, chunk) batches; strides of (head, chunk, row, column)
// for each operand; m/n/k_chunk: that dimension is the chunk's (ragged last chunk);
// lower: only the lower triangle of C (with the diagonal) is formed.
struct ChunkGemm {
  int heads, chunks, chunk, seq;
  hipStream_t s;
  hipError_t operator()(const float* A, int64_t ah, int64_t ac, int64_t ai, int64_t ak, const float* Bm, int64_t bh,
                        int64_t bc, int64_t bk, int64_t bj, float* Cm, int64_t ch, int64_t c2, int64_t ci, int64_t cj,
                        int Mm, int Nn, int Kk, int mc, int nc, int kc, int lower, int acc) const {
    luna::BwdGemm g{};
    g.A = A; g.sAh = ah; g.sAc = ac; g.sAi = ai; g.sAk = ak;
    g.B = Bm; g.sBh = bh; g.sBc = bc; g.sBk = bk; g.sBj = bj;
    g.C = Cm; g.sCh = ch; g.sCc = c2; g.sCi = ci; g.sCj = cj;
    g.M = Mm; g.N = Nn; g.K = Kk;
    g.heads = heads; g.chunks = chunks; g.chunk = chunk; g.seq = seq;
    g.m_chunk = mc; g.n_chunk = nc; g.k_chunk = kc; g.lower = lower; g.accumulate = acc;
    return luna::launch_bwd_gemm(g, s);
  }
};

// The attention part of the fp32 forward for given fp32 features (eq. (9) of
// Section 3.1, the causal form in 64-token chunks): [V | 1], per-chunk [S_c | z_c] =
// phi(K_c)^T [V_c | 1], their exclusive prefix over chunks (causal) or total, and with
// queries [num | den - eps] = phi(Q_c) [S_c | z_c] (+ P_c [V_c | 1], P_c =
// tril(phi(Q_c) phi(K_c)^T)).  phiq == nullptr: the state only.
luna_status enqueue_f32_attention(luna::Dt vdt, int64_t heads64, int64_t n, int dd, int D, uint8_t* w,
                                  const Layout& lay, const float* phiq, const float* phik, const void* V, bool causal,
                                  hipStream_t s) {
  const int heads = (int)heads64, E = dd + 1, C = lay.chunk, nch = lay.nch;
  const int64_t nD = n * D, nE = n * E, st_el = (int64_t)D * E, cc = (int64_t)C * C;
  float* vx = reinterpret_cast<float*>(w + lay.vx);
  float* y = reinterpret_cast<float*>(w + lay.y);
  float* sx = reinterpret_cast<float*>(w + lay.sx);
  float* pm = reinterpret_cast<float*>(w + lay.pm);
  hipError_t e;
#define LUNA_TRY(expr, what) \
  if ((e = (expr)) != hipSuccess) return hip_fail(e, what)
  LUNA_TRY(luna::launch_bwd_pack(vdt, V, vx, heads64 * n, dd, s), "pack kernel launch");
  const ChunkGemm gemm{heads, nch, C, (int)n, s};
  const int64_t sh = (int64_t)nch * st_el;  // head stride of the per-chunk states
  LUNA_TRY(gemm(phik, nD, (int64_t)C * D, 1, D, vx, nE, (int64_t)C * E, E, 1, sx, sh, st_el, E, 1, D, E, C, 0, 0, 1,
                0, 0), "state GEMM");
  LUNA_TRY(luna::launch_bwd_scan(sx, heads, nch, st_el, causal ? 0 : 2, s), "state scan");
  if (!phiq) return LUNA_OK;
  LUNA_TRY(gemm(phiq, nD, (int64_t)C * D, D, 1, sx, sh, st_el, E, 1, y, nE, (int64_t)C * E, E, 1, C, E, D, 1, 0, 0,
                0, 0), "readout GEMM");
  if (causal) {
    LUNA_TRY(gemm(phiq, nD, (int64_t)C * D, D, 1, phik, nD, (int64_t)C * D, 1, D, pm, nch * cc, cc, C, 1, C, C, D, 1,
                  1, 0, 1, 0), "P GEMM");
    LUNA_TRY(gemm(pm, nch * cc, cc, C, 1, vx, nE, (int64_t)C * E, E, 1, y, nE, (int64_t)C * E, E, 1, C, E, C, 1, 0,
                  1, 0, 1), "intra-chunk GEMM");
  }
#undef LUNA_TRY
  return LUNA_OK;
}

// The forward pass in fp32: features of the keys (and queries) by the feature-map
// kernel, then enqueue_f32_attention.  Q == nullptr: the state only.
luna_status enqueue_f32_forward(const Problem& pb, uint8_t* w, const Layout& lay, const void* Q, const void* K,
                                const void* V, bool causal, hipStream_t s) {
  const luna::Dt dt = pb.dt == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int L = pb.p->L, D = pb.p->M * L, dd = (int)pb.d;
  float* phiq = reinterpret_cast<float*>(w + lay.phiq);
  float* phik = reinterpret_cast<float*>(w + lay.phik);
  luna::FeatureMapArgs f{};  // queries and keys in one launch
  f.phi = phi_args(pb, w, lay);
  f.rows_per_head = pb.n;
  f.H = (int)pb.H;
  f.heads = pb.B * pb.H;
  f.X = K;
  f.out = phik;
  if (Q) {
    f.X2 = Q;
    f.out2 = phiq;
  }
  const hipError_t e = luna::launch_featuremap(dt, luna::Dt::F32, dd, L, f, s);
  if (e != hipSuccess) return hip_fail(e, "feature-map kernel launch");
  return enqueue_f32_attention(dt, pb.B * pb.H, pb.n, dd, D, w, lay, Q ? phiq : nullptr, phik, V, causal, s);
}

// The generic forward: the fp32 forward, then out = num / den in the call's dtype.
luna_status enqueue_generic_attn(const Problem& pb, uint8_t* w, const Layout& lay, const void* Q, const void* K,
                                 const void* V, float eps, void* out, bool causal, hipStream_t s) {
  luna_status st = enqueue_f32_forward(pb, w, lay, Q, K, V, causal, s);
  if (st != LUNA_OK) return st;
  const hipError_t e = luna::launch_fwd_out(pb.dt == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32,
                                            reinterpret_cast<const float*>(w + lay.y), out, pb.B * pb.H * pb.n,
                                            (int)pb.d, eps, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "output kernel launch");
}

// Scratch of luna_attn_fwd_causal_noalloc: one array per device, part of the code
// object, so that calls need no allocation.  Host code never uses the array's name as
// an address (on the host it only stands in for the symbol): the device address comes
// from hipGetSymbolAddress, once per device, and is kept here.
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) uint8_t scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch.
luna_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(LUNA_ERR_UNSUPPORTED, "device index must be below 64");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress of the scratch array");
    if (ptr == nullptr || ((uintptr_t)ptr & 255) != 0) return fail(LUNA_ERR_HIP, "scratch array address not 256-byte aligned");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return LUNA_OK;
}

// A variant description's features per row (D) after checking it completely.
luna_status check_variant(const luna_phi_variant* v, int64_t* D) {
  if (v == nullptr || v->base == nullptr) return fail(LUNA_ERR_INVALID_ARG, "variant or its base parameters is NULL");
  const luna_phi_params* p = v->base;
  if (v->kind < LUNA_PHI_MLP || v->kind > LUNA_PHI_PERFORMER) return fail(LUNA_ERR_INVALID_ARG, "unknown variant kind");
  if (p->M < 1 || p->M > 256) return fail(LUNA_ERR_INVALID_ARG, "M must be in [1, 256]");
  if (p->per_head != 0 && p->per_head != 1) return fail(LUNA_ERR_INVALID_ARG, "per_head must be 0 or 1");
  if (!p->W || !p->b) return fail(LUNA_ERR_INVALID_ARG, "W or b is NULL");
  if ((v->env_w == nullptr) != (v->env_b == nullptr)) return fail(LUNA_ERR_INVALID_ARG, "env_w and env_b go together");
  if (v->ch_rms != 0 && v->ch_rms != 1) return fail(LUNA_ERR_INVALID_ARG, "ch_rms must be 0 or 1");
  if (v->kind != LUNA_PHI_MLP) {
    if (v->env_w || v->bank || v->ch_rms)
      return fail(LUNA_ERR_INVALID_ARG, "an envelope, bank or channel RMS needs the channel-MLP kind");
    *D = v->kind == LUNA_PHI_RFF_SINCOS ? 2 * (int64_t)p->M : p->M;
    return LUNA_OK;
  }
  if (v->act < LUNA_ACT_RELU || v->act > LUNA_ACT_TANH) return fail(LUNA_ERR_INVALID_ARG, "unknown activation");
  if (p->L < 1 || p->L > 16) return fail(LUNA_ERR_INVALID_ARG, "L must be in [1, 16]");
  if (p->hidden < 1 || p->hidden > 64) return fail(LUNA_ERR_INVALID_ARG, "hidden must be in [1, 64]");
  if (p->shared_channels != 0 && p->shared_channels != 1) return fail(LUNA_ERR_INVALID_ARG, "shared_channels must be 0 or 1");
  if (p->nonneg != 0 && p->nonneg != 1) return fail(LUNA_ERR_INVALID_ARG, "nonneg must be 0 or 1");
  if (!p->fc1_w || !p->fc1_b || !p->fc2_w || !p->fc2_b) return fail(LUNA_ERR_INVALID_ARG, "a channel-MLP array is NULL");
  if (v->ch_rms && !(std::isfinite(v->ch_rms_target) && v->ch_rms_target > 0.0f))
    return fail(LUNA_ERR_INVALID_ARG, "ch_rms_target must be finite and > 0");
  *D = v->bank ? (int64_t)p->M : (int64_t)p->M * p->L;
  if (*D > 512) return fail(LUNA_ERR_INVALID_ARG, "a variant has at most 512 features");
  return LUNA_OK;
}

// Workspace of a variant map of `rows` rows: with channel RMS, the per-workgroup
// partial sums, the channel scales and y of every row in fp32 ([row][M][L]).
constexpr size_t kVarPartialBytes = (size_t)luna::kVariantMaxGrid * luna::kVariantMaxL * sizeof(double);
constexpr size_t kVarScaleBytes = 256;
size_t variant_ws_bytes(const luna_phi_variant* v, int64_t rows) {
  if (v->kind != LUNA_PHI_MLP || !v->ch_rms) return 0;
  return align256(kVarPartialBytes) + kVarScaleBytes +
         align256((size_t)rows * (size_t)v->base->M * (size_t)v->base->L * sizeof(float));
}

// Buffers of luna_attn_fwd_features: the causal scan kernel on the bf16 features when
// it is built for (d, D), else the fp32 GEMM path (fp32 copies of bf16 features).
luna_status plan_features(luna_dtype phi_dtype, luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                          int64_t D, int32_t causal, int32_t chunk, Layout* lay) {
  if ((phi_dtype != LUNA_F32 && phi_dtype != LUNA_BF16) || (dtype != LUNA_F32 && dtype != LUNA_BF16))
    return fail(LUNA_ERR_INVALID_ARG, "dtypes must be LUNA_F32 or LUNA_BF16");
  if (B < 1 || H < 1 || n < 1) return fail(LUNA_ERR_INVALID_ARG, "B, H and n must be >= 1");
  if (n > (int64_t)1 << 30 || B * H > (int64_t)1 << 24) return fail(LUNA_ERR_UNSUPPORTED, "n or B*H too large");
  if (d < 1 || d > 256) return fail(LUNA_ERR_UNSUPPORTED, "d must be in [1, 256]");
  if (D < 1 || D > 512) return fail(LUNA_ERR_UNSUPPORTED, "D must be in [1, 512]");
  if (causal != 0 && causal != 1) return fail(LUNA_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (causal && chunk != 64) return fail(LUNA_ERR_UNSUPPORTED, "chunk must be 64");
  const int64_t heads = B * H;
  size_t off = 0;
  if (causal && phi_dtype == LUNA_BF16 && dtype == LUNA_BF16 && luna::causal_given_supported(luna::Dt::BF16, (int)d, (int)D)) {
    lay->given = 1;
    plan_causal_parts(heads, n, luna::causal_given_state_floats((int)d, (int)D), lay, &off, false);
  } else {
    lay->generic = 1;
    luna_status st = plan_f32_buffers(heads, n, (int)d, (int)D, causal != 0, true, phi_dtype == LUNA_BF16, lay, &off);
    if (st != LUNA_OK) return st;
  }
  lay->total = off;
  return LUNA_OK;
}

// Through the feature map, from dphi(Q) and dphi(K) in the workspace (fp32, [head][n][D]):
// u = [x | 1] [W | b]^T (GEMM), du from dphi on the tables, [dW | db] = du^T [x | 1]
// and the channel-MLP gradients into grads (when given), dx = du [W | b] into dQ, dK
// (when given).  Used by the backward pass and by the distillation loss.
luna_status enqueue_phi_backward(const Problem& pb, uint8_t* w, const Layout& lay, const void* Q, const void* K,
                                 void* dQ, void* dK, const luna_phi_grads* grads, hipStream_t s) {
  const luna_phi_params* p = pb.p;
  const luna::Dt dt = pb.dt == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int64_t B = pb.B, H = pb.H, n = pb.n;
  const int M = p->M, L = p->L, dd = (int)pb.d, E = dd + 1;
  const int heads = (int)(B * H);
  const int64_t nE = n * E;
  float* dphiq = reinterpret_cast<float*>(w + lay.dphiq);
  float* dphik = reinterpret_cast<float*>(w + lay.dphik);
  hipError_t e;
#define LUNA_TRY(expr, what) \
  if ((e = (expr)) != hipSuccess) return hip_fail(e, what)
  const int P = param_sets(pb);
  const int Hh = (int)H, Bb = (int)B;
  float* xq = reinterpret_cast<float*>(w + lay.xq);
  float* xk = reinterpret_cast<float*>(w + lay.xk);
  float* wx = reinterpret_cast<float*>(w + lay.wx);
  float* uq = reinterpret_cast<float*>(w + lay.uq);
  float* uk = reinterpret_cast<float*>(w + lay.uk);
  float* duq = reinterpret_cast<float*>(w + lay.duq);
  float* duk = reinterpret_cast<float*>(w + lay.duk);
  float* dwh = reinterpret_cast<float*>(w + lay.dwh);
  LUNA_TRY(luna::launch_bwd_pack(dt, Q, xq, (int64_t)heads * n, dd, s), "pack kernel launch");
  LUNA_TRY(luna::launch_bwd_pack(dt, K, xk, (int64_t)heads * n, dd, s), "pack kernel launch");
  LUNA_TRY(luna::launch_bwd_packw(dt, p->W, p->b, wx, P * M, dd, s), "pack kernel launch");
  // products over (batch, head) pairs: the batch index is the GEMM's head, the head its
  // chunk, so that per-head parameters are addressed by stride
  const int64_t wsc = p->per_head ? (int64_t)M * E : 0;
  auto gemm_bh = [&](const float* A, int64_t ah, int64_t ac, int64_t ai, int64_t ak, const float* Bm, int64_t bh,
                     int64_t bc, int64_t bk, int64_t bj, float* Cm, int64_t ch, int64_t c2, int64_t ci, int64_t cj, int Mm,
                     int Nn, int Kk, int acc) {
    luna::BwdGemm g{};
    g.A = A; g.sAh = ah; g.sAc = ac; g.sAi = ai; g.sAk = ak;
    g.B = Bm; g.sBh = bh; g.sBc = bc; g.sBk = bk; g.sBj = bj;
    g.C = Cm; g.sCh = ch; g.sCc = c2; g.sCi = ci; g.sCj = cj;
    g.M = Mm; g.N = Nn; g.K = Kk;
    g.heads = Bb; g.chunks = Hh; g.chunk = (int)n; g.seq = (int)n;
    g.accumulate = acc;
    return luna::launch_bwd_gemm(g, s);
  };
  const int64_t nM = n * M, ME = (int64_t)M * E;
  for (int side = 0; side < 2; ++side) {
    const float* x = side ? xk : xq;
    float* u = side ? uk : uq;
    LUNA_TRY(gemm_bh(x, Hh * nE, nE, E, 1, wx, 0, wsc, 1, E, u, Hh * nM, nM, M, 1, (int)n, M, E, 0), "projection GEMM");
  }
  luna::BwdPhi ph{};
  ph.uq = uq;
  ph.uk = uk;
  ph.dphiq = dphiq;
  ph.dphik = dphik;
  ph.duq = duq;
  ph.duk = duk;
  ph.tables = w + lay.tables;
  ph.partial = reinterpret_cast<float*>(w + lay.bpart);
  ph.n = n;
  ph.heads = B * H;
  ph.H = Hh;
  ph.M = M;
  ph.per_head = p->per_head;
  ph.part_floats = lay.part_floats;
  LUNA_TRY(luna::launch_bwd_phi(L, ph, lay.groups, P, s), "feature-map backward kernel launch");
  for (int side = 0; side < 2; ++side) {
    float* x = side ? xk : xq;
    const float* du = side ? duk : duq;
    if (grads)  // [dW | db] per (batch, head), both sides added
      LUNA_TRY(gemm_bh(du, Hh * nM, nM, 1, M, x, Hh * nE, nE, E, 1, dwh, Hh * ME, ME, E, 1, M, E, (int)n, side),
               "weight-gradient GEMM");
    // dx = du [W | b] into x's rows (x is not read again), then its first d columns
    void* dx = side ? dK : dQ;
    if (dx == nullptr) continue;
    LUNA_TRY(gemm_bh(du, Hh * nM, nM, M, 1, wx, 0, wsc, E, 1, x, Hh * nE, nE, E, 1, (int)n, E, M, 0), "dx GEMM");
    LUNA_TRY(luna::launch_bwd_cols(dt, x, dx, (int64_t)heads * n, dd, s), "dx convert");
  }
  if (grads) {
    LUNA_TRY(luna::launch_bwd_dw(dwh, grads->W, grads->b, Bb, Hh, M, dd, p->per_head, s), "weight-gradient sum");
    const int units = (p->shared_channels ? 1 : L) * p->hidden;
    const int used = 2 * (units + 1) * L;
    double* sum = reinterpret_cast<double*>(w + lay.sum);
    double* pre = reinterpret_cast<double*>(w + lay.pre);
    LUNA_TRY(luna::launch_bwd_reduce(ph.partial, sum, lay.groups, lay.part_floats, used, P, s), "reduce kernel launch");
    LUNA_TRY(luna::launch_bwd_prefix(sum, pre, w + lay.tables, M, dd, L, lay.part_floats, luna::bwd_nseg_cap(L), P, s),
             "prefix kernel launch");
    luna::BwdMlp m{};
    m.sum = sum;
    m.pre = pre;
    m.tables = w + lay.tables;
    m.fc1_w = p->fc1_w;
    m.fc1_b = p->fc1_b;
    m.fc2_w = p->fc2_w;
    m.dfc1_w = grads->fc1_w;
    m.dfc1_b = grads->fc1_b;
    m.dfc2_w = grads->fc2_w;
    m.dfc2_b = grads->fc2_b;
    m.L = L;
    m.hidden = p->hidden;
    m.C1 = p->shared_channels ? 1 : L;
    m.part_floats = lay.part_floats;
    m.nseg_cap = luna::bwd_nseg_cap(L);
    LUNA_TRY(luna::launch_bwd_mlp(m, P, s), "parameter-gradient kernel launch");
  }
#undef LUNA_TRY
  return LUNA_OK;
}

}  // namespace

extern "C" {

int64_t luna_phi_variant_features(const luna_phi_variant* v) {
  int64_t D = -1;
  return check_variant(v, &D) == LUNA_OK ? D : -1;
}

size_t luna_featuremap_variant_workspace_bytes(luna_dtype, int64_t B, int64_t H, int64_t n, int64_t,
                                               const luna_phi_variant* v) {
  int64_t D = 0;
  if (B < 1 || H < 1 || n < 1 || n > (int64_t)1 << 30 || B * H > (int64_t)1 << 24) return 0;
  return check_variant(v, &D) == LUNA_OK ? variant_ws_bytes(v, B * H * n) : 0;
}

luna_status luna_featuremap_variant(const void* X, luna_dtype x_dtype, int64_t B, int64_t H, int64_t n,
                                    int64_t d, const luna_phi_variant* v, void* phi_out, luna_dtype out_dtype,
                                    void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  int64_t D = 0;
  luna_status st = check_variant(v, &D);
  if (st != LUNA_OK) return st;
  if ((x_dtype != LUNA_F32 && x_dtype != LUNA_BF16) || (out_dtype != LUNA_F32 && out_dtype != LUNA_BF16))
    return fail(LUNA_ERR_INVALID_ARG, "dtypes must be LUNA_F32 or LUNA_BF16");
  if (B < 1 || H < 1 || n < 1) return fail(LUNA_ERR_INVALID_ARG, "B, H and n must be >= 1");
  if (n > (int64_t)1 << 30 || B * H > (int64_t)1 << 24) return fail(LUNA_ERR_UNSUPPORTED, "n or B*H too large");
  if (d != 32 && d != 64 && d != 128) return fail(LUNA_ERR_UNSUPPORTED, "d must be 32, 64 or 128");
  if (!X || !phi_out) return fail(LUNA_ERR_INVALID_ARG, "X or phi_out is NULL");
  const size_t need = variant_ws_bytes(v, B * H * n);
  if (need) {
    Layout lay;
    lay.total = need;
    if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  }
  const luna_phi_params* p = v->base;
  luna::VariantArgs a{};
  a.X = X;
  a.out = phi_out;
  a.W = p->W;
  a.b = p->b;
  a.kind = v->kind;
  a.M = p->M;
  a.per_head = p->per_head;
  a.H = (int)H;
  a.rows_per_head = n;
  a.heads = B * H;
  a.L = 1;
  a.hidden = 1;
  a.C1 = 1;
  if (v->kind == LUNA_PHI_MLP) {
    a.act = v->act;
    a.L = p->L;
    a.hidden = p->hidden;
    a.C1 = p->shared_channels ? 1 : p->L;
    a.nonneg = p->nonneg;
    a.fc1_w = p->fc1_w;
    a.fc1_b = p->fc1_b;
    a.fc2_w = p->fc2_w;
    a.fc2_b = p->fc2_b;
    a.env_w = v->env_w;
    a.env_b = v->env_b;
    a.bank = v->bank;
  }
  const luna::Dt idt = x_dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  a.out_bf16 = out_dtype == LUNA_BF16;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e;
  int grid = 0;
  if (need) {  // channel RMS: y and the sums of y^2, the scales, then phi from y
    uint8_t* w = static_cast<uint8_t*>(ws);
    double* partial = reinterpret_cast<double*>(w);
    float* scale = reinterpret_cast<float*>(w + align256(kVarPartialBytes));
    a.rms_pass = 1;
    a.rms_partial = partial;
    a.rms_y = reinterpret_cast<float*>(w + align256(kVarPartialBytes) + kVarScaleBytes);
    if ((e = luna::launch_variant_map(idt, (int)d, a, &grid, s)) != hipSuccess) return hip_fail(e, "variant map launch");
    const double count = (double)(B * H) * (double)n * (double)p->M;
    if ((e = luna::launch_variant_rms(partial, grid, p->L, count, v->ch_rms_target, scale, s)) != hipSuccess)
      return hip_fail(e, "channel RMS kernel launch");
    e = luna::launch_variant_finish(a, scale, s);
    return e == hipSuccess ? LUNA_OK : hip_fail(e, "channel RMS output kernel launch");
  }
  e = luna::launch_variant_map(idt, (int)d, a, &grid, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "variant map launch");
}

size_t luna_attn_features_workspace_bytes(luna_dtype phi_dtype, luna_dtype dtype, int64_t B, int64_t H, int64_t n,
                                          int64_t d, int64_t D, int32_t causal, int32_t chunk) {
  Layout lay;
  return plan_features(phi_dtype, dtype, B, H, n, d, D, causal, chunk, &lay) == LUNA_OK ? lay.total : 0;
}

luna_status luna_attn_fwd_features(const void* phiQ, const void* phiK, luna_dtype phi_dtype, const void* V,
                                   luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d, int64_t D,
                                   int32_t causal, int32_t chunk, float eps, void* out, void* ws, size_t ws_bytes,
                                   void* stream) {
  g_last_error.clear();
  Layout lay;
  luna_status st = plan_features(phi_dtype, dtype, B, H, n, d, D, causal, chunk, &lay);
  if (st != LUNA_OK) return st;
  if (!phiQ || !phiK || !V || !out) return fail(LUNA_ERR_INVALID_ARG, "phiQ, phiK, V or out is NULL");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (lay.total && (st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  const luna::Dt vdt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  hipError_t e;
  if (lay.given) {  // the causal scan kernel on the bf16 features
    luna::CausalArgs a{};
    a.Q = phiQ;
    a.K = phiK;
    a.V = V;
    a.out = out;
    a.phi.M = (int)D;
    a.n = (int)n;
    a.H = (int)H;
    a.heads = (int)(B * H);
    a.parts = lay.parts;
    a.split = lay.split;
    a.eps = eps;
    a.phiq = phiQ;
    a.phik = phiK;
    if (lay.parts == 2) {
      float* stp = reinterpret_cast<float*>(w + lay.state);
      a.pieces = lay.pieces;
      a.piece_chunks = lay.piece_chunks;
      a.state_out = stp;
      if ((e = luna::launch_causal_given((int)d, (int)D, a, s)) != hipSuccess) return hip_fail(e, "state launch");
      a.state_out = nullptr;
      a.state_in = stp;
    }
    e = luna::launch_causal_given((int)d, (int)D, a, s);
    return e == hipSuccess ? LUNA_OK : hip_fail(e, "causal attention kernel launch");
  }
  const int64_t heads = B * H;
  const float* fq = static_cast<const float*>(phiQ);
  const float* fk = static_cast<const float*>(phiK);
  if (phi_dtype == LUNA_BF16) {  // fp32 copies of the features
    float* q32 = reinterpret_cast<float*>(w + lay.phiq);
    float* k32 = reinterpret_cast<float*>(w + lay.phik);
    if ((e = luna::launch_widen(luna::Dt::BF16, phiQ, q32, heads * n * D, s)) != hipSuccess) return hip_fail(e, "widen");
    if ((e = luna::launch_widen(luna::Dt::BF16, phiK, k32, heads * n * D, s)) != hipSuccess) return hip_fail(e, "widen");
    fq = q32;
    fk = k32;
  }
  if ((st = enqueue_f32_attention(vdt, heads, n, (int)d, (int)D, w, lay, fq, fk, V, causal != 0, s)) != LUNA_OK)
    return st;
  e = luna::launch_fwd_out(vdt, reinterpret_cast<const float*>(w + lay.y), out, heads * n, (int)d, eps, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "output kernel launch");
}


size_t luna_workspace_bytes(int32_t op, luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                            const luna_phi_params* p, int32_t chunk) {
  Problem pb{op, dtype, B, H, n, d, p, chunk};
  Layout lay;
  return plan(pb, &lay) == LUNA_OK ? lay.total : 0;
}

luna_status luna_featuremap(const void* X, luna_dtype x_dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                            const luna_phi_params* p, void* phi_out, luna_dtype out_dtype, void* ws,
                            size_t ws_bytes, void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_FEATUREMAP, x_dtype, B, H, n, d, p, 0};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (out_dtype != LUNA_F32 && out_dtype != LUNA_BF16) return fail(LUNA_ERR_INVALID_ARG, "out_dtype must be LUNA_F32 or LUNA_BF16");
  if (!X || !phi_out) return fail(LUNA_ERR_INVALID_ARG, "X or phi_out is NULL");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  luna::FeatureMapArgs a{};
  a.X = X;
  a.out = phi_out;
  a.phi = phi_args(pb, w, lay);
  a.rows_per_head = n;
  a.H = (int)H;
  a.heads = B * H;
  hipError_t e = luna::launch_featuremap(x_dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32,
                                         out_dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32, (int)d, p->L, a, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "feature-map kernel launch");
}

luna_status luna_attn_fwd(const void* Q, const void* K, const void* V, luna_dtype dtype, int64_t B, int64_t H,
                          int64_t n, int64_t d, const luna_phi_params* p, float eps, void* out, void* ws,
                          size_t ws_bytes, void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_ATTN, dtype, B, H, n, d, p, 0};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!Q || !K || !V || !out) return fail(LUNA_ERR_INVALID_ARG, "Q, K, V or out is NULL");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  if (lay.generic) return enqueue_generic_attn(pb, w, lay, Q, K, V, eps, out, false, s);
  luna::NoncausalArgs a{};
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.out = out;
  a.phi = phi_args(pb, w, lay);
  a.n = (int)n;
  a.H = (int)H;
  a.heads = (int)(B * H);
  a.splits = lay.splits;
  a.tokens_per_split = lay.tokens_per_split;
  a.eps = eps;
  a.partial = reinterpret_cast<float*>(w + lay.partial);
  a.frags = w + lay.frags;
  a.tile_tokens = lay.tile_tokens;
  a.tiles = lay.tiles;
  a.fused = lay.fused;
  hipError_t e = luna::launch_noncausal(dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32, (int)d, p->L, p->M, a, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "attention kernel launch");
}

luna_status luna_attn_fwd_causal(const void* Q, const void* K, const void* V, luna_dtype dtype, int64_t B,
                                 int64_t H, int64_t n, int64_t d, const luna_phi_params* p, int32_t chunk, float eps,
                                 void* out, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_ATTN_CAUSAL, dtype, B, H, n, d, p, chunk};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!Q || !K || !V || !out) return fail(LUNA_ERR_INVALID_ARG, "Q, K, V or out is NULL");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  if (lay.generic) return enqueue_generic_attn(pb, w, lay, Q, K, V, eps, out, true, s);
  luna::CausalArgs a{};
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.out = out;
  a.phi = phi_args(pb, w, lay);
  a.n = (int)n;
  a.H = (int)H;
  a.heads = (int)(B * H);
  a.parts = lay.parts;
  a.split = lay.split;
  a.eps = eps;
  const luna::Dt dt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int D = p->M * p->L;
  if (lay.given) {  // phi(Q), phi(K) in bf16 first (one launch)
    luna::FeatureMapArgs f{};
    f.phi = a.phi;
    f.rows_per_head = n;
    f.H = (int)H;
    f.heads = B * H;
    f.X = Q;
    f.out = w + lay.phiq;
    f.X2 = K;
    f.out2 = w + lay.phik;
    hipError_t e = luna::launch_featuremap(dt, luna::Dt::BF16, (int)d, p->L, f, s);
    if (e != hipSuccess) return hip_fail(e, "feature-map kernel launch");
    a.phiq = w + lay.phiq;
    a.phik = w + lay.phik;
  }
  auto launch = [&]() {
    return lay.given ? luna::launch_causal_given((int)d, D, a, s) : luna::launch_causal(dt, (int)d, p->L, p->M, a, s);
  };
  if (lay.staged) {
    // launch 1: part 0 scans [0, A), part 1 sums the state of [A, A + B); both write
    // their final states as pieces 0 and 1.  launch 2: part 0 scans [A, A + B) from
    // piece 0, part 1 scans [A + B, nch) from pieces 0 + 1.
    const int A = lay.sa, AB = lay.sa + lay.sb, nch = (int)((n + 63) / 64);
    float* st = reinterpret_cast<float*>(w + lay.state);
    a.staged = 1;
    a.pieces = 2;
    a.pc_first[0] = 0;  a.pc_begin[0] = 0;  a.pc_end[0] = A;  a.pseed[0] = 0;
    a.pc_first[1] = A;  a.pc_begin[1] = AB; a.pc_end[1] = AB; a.pseed[1] = 0;
    a.state_fin = st;
    hipError_t e = launch();
    if (e != hipSuccess) return hip_fail(e, "causal attention first scan launch");
    a.pc_first[0] = A;  a.pc_begin[0] = A;  a.pc_end[0] = AB;  a.pseed[0] = 1;
    a.pc_first[1] = AB; a.pc_begin[1] = AB; a.pc_end[1] = nch; a.pseed[1] = 2;
    a.state_fin = nullptr;
    a.state_in = st;
    e = launch();
    return e == hipSuccess ? LUNA_OK : hip_fail(e, "causal attention second scan launch");
  }
  if (lay.parts == 2) {
    float* st = reinterpret_cast<float*>(w + lay.state);
    a.pieces = lay.pieces;
    a.piece_chunks = lay.piece_chunks;
    a.state_out = st;
    hipError_t e = launch();
    if (e != hipSuccess) return hip_fail(e, "causal attention state launch");
    a.state_out = nullptr;
    a.state_in = st;
  }
  hipError_t e = launch();
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "causal attention kernel launch");
}

luna_status luna_attn_fwd_causal_noalloc(const void* Q, const void* K, const void* V, luna_dtype dtype,
                                         int64_t B, int64_t H, int64_t n, int64_t d, const luna_phi_params* p,
                                         int32_t chunk, float eps, void* out, void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_ATTN_CAUSAL, dtype, B, H, n, d, p, chunk};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (lay.total > kScratchBytes) {
    char buf[160];
    snprintf(buf, sizeof buf, "problem needs %zu bytes of scratch; the static scratch holds %zu", lay.total,
             kScratchBytes);
    return fail(LUNA_ERR_WORKSPACE, buf);
  }
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != LUNA_OK) return st;
  return luna_attn_fwd_causal(Q, K, V, dtype, B, H, n, d, p, chunk, eps, out, ws, kScratchBytes, stream);
}

size_t luna_noalloc_scratch_bytes(void) { return kScratchBytes; }

luna_status luna_attn_state(const void* K, const void* V, luna_dtype dtype, int64_t B, int64_t H, int64_t n,
                            int64_t d, const luna_phi_params* p, int32_t accumulate, float* S, float* z, void* ws,
                            size_t ws_bytes, void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_STATE, dtype, B, H, n, d, p, 0};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!K || !V || !S || !z) return fail(LUNA_ERR_INVALID_ARG, "K, V, S or z is NULL");
  if (accumulate != 0 && accumulate != 1) return fail(LUNA_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  const luna::Dt dt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  if (lay.generic) {
    if ((st = enqueue_f32_forward(pb, w, lay, nullptr, K, V, false, s)) != LUNA_OK) return st;
    // every piece holds the total after the scan: export the first
    const int D = p->M * p->L;
    const hipError_t e = luna::launch_fwd_export(reinterpret_cast<const float*>(w + lay.sx),
                                                 (int64_t)lay.nch * D * (d + 1), S, z, (int)(B * H), D, (int)d,
                                                 accumulate, s);
    return e == hipSuccess ? LUNA_OK : hip_fail(e, "state export kernel launch");
  }
  if (lay.pieces == 0) {
    luna::NoncausalArgs a{};
    a.K = K;
    a.V = V;
    a.phi = phi_args(pb, w, lay);
    a.n = (int)n;
    a.H = (int)H;
    a.heads = (int)(B * H);
    a.splits = lay.splits;
    a.tokens_per_split = lay.tokens_per_split;
    a.partial = reinterpret_cast<float*>(w + lay.partial);
    a.state_S = S;
    a.state_z = z;
    a.accumulate = accumulate;
    hipError_t e = luna::launch_state(dt, (int)d, p->L, p->M, a, s);
    return e == hipSuccess ? LUNA_OK : hip_fail(e, "state kernel launch");
  }
  luna::CausalArgs a{};
  a.K = K;
  a.V = V;
  a.Q = K;  // (the state launch reads no query rows)
  a.phi = phi_args(pb, w, lay);
  a.n = (int)n;
  a.H = (int)H;
  a.heads = (int)(B * H);
  a.parts = 2;
  a.split = lay.split;
  a.pieces = lay.pieces;
  a.piece_chunks = lay.piece_chunks;
  a.state_out = reinterpret_cast<float*>(w + lay.state);
  hipError_t e = luna::launch_causal(dt, (int)d, p->L, p->M, a, s);
  if (e != hipSuccess) return hip_fail(e, "causal state launch");
  a.export_S = S;
  a.export_z = z;
  a.accumulate = accumulate;
  e = luna::launch_causal(dt, (int)d, p->L, p->M, a, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "state export launch");
}

luna_status luna_attn_causal_step(const void* Q, const void* K, const void* V, luna_dtype dtype, int64_t B,
                                  int64_t H, int64_t m, int64_t d, const luna_phi_params* p, float eps,
                                  int32_t tables_ready, float* S, float* z, void* out, void* ws, size_t ws_bytes,
                                  void* stream) {
  g_last_error.clear();
  Problem pb{LUNA_OP_CAUSAL_STEP, dtype, B, H, m, d, p, 0};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!Q || !K || !V || !S || !z || !out) return fail(LUNA_ERR_INVALID_ARG, "Q, K, V, S, z or out is NULL");
  if (((uintptr_t)S & 15) != 0) return fail(LUNA_ERR_INVALID_ARG, "S must be 16-byte aligned");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (tables_ready != 0 && tables_ready != 1) return fail(LUNA_ERR_INVALID_ARG, "tables_ready must be 0 or 1");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if (!tables_ready && (st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  const luna::Dt dt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  luna::FeatureMapArgs f{};  // queries and keys in one launch
  f.phi = phi_args(pb, w, lay);
  f.rows_per_head = m;
  f.H = (int)H;
  f.heads = B * H;
  if (!p->per_head && B * H * m <= ((int64_t)1 << 30)) {
    // one parameter set: the rows of all heads are one contiguous array, mapped in
    // 64-row tiles across heads (a one-token step then needs B*H/64 tiles, not B*H)
    f.rows_per_head = B * H * m;
    f.H = 1;
    f.heads = 1;
  }
  f.X = Q;
  f.out = w + lay.phiq;
  f.X2 = K;
  f.out2 = w + lay.phik;
  // z before the step, for every column block of a head to read (block 0 rewrites z),
  // copied by workgroups of the same launch
  f.copy_src = z;
  f.copy_dst = reinterpret_cast<float*>(w + lay.zcopy);
  f.copy_n = (B * H) * (int64_t)(p->M * p->L);
  hipError_t e = luna::launch_featuremap(dt, luna::Dt::F32, (int)d, p->L, f, s);
  if (e != hipSuccess) return hip_fail(e, "feature-map kernel launch");
  luna::StepArgs a{};
  a.phiq = reinterpret_cast<const float*>(w + lay.phiq);
  a.phik = reinterpret_cast<const float*>(w + lay.phik);
  a.V = V;
  a.out = out;
  a.S = S;
  a.z = z;
  a.z_in = reinterpret_cast<const float*>(w + lay.zcopy);
  a.m = (int)m;
  a.d = (int)d;
  a.D = p->M * p->L;
  a.heads = (int)(B * H);
  a.eps = eps;
  e = luna::launch_causal_step(dt, a, s);
  return e == hipSuccess ? LUNA_OK : hip_fail(e, "streaming step kernel launch");
}

luna_status luna_attn_bwd(const void* Q, const void* K, const void* V, const void* dO, luna_dtype dtype, int64_t B,
                          int64_t H, int64_t n, int64_t d, const luna_phi_params* p, int32_t causal, float eps,
                          void* dQ, void* dK, void* dV, const luna_phi_grads* grads, void* ws, size_t ws_bytes,
                          void* stream) {
  g_last_error.clear();
  if (causal != 0 && causal != 1) return fail(LUNA_ERR_INVALID_ARG, "causal must be 0 or 1");
  Problem pb{causal ? LUNA_OP_ATTN_CAUSAL_BWD : LUNA_OP_ATTN_BWD, dtype, B, H, n, d, p, 64};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!Q || !K || !V || !dO || !dQ || !dK || !dV) return fail(LUNA_ERR_INVALID_ARG, "an input or output is NULL");
  if (grads && (!grads->W || !grads->b || !grads->fc1_w || !grads->fc1_b || !grads->fc2_w || !grads->fc2_b))
    return fail(LUNA_ERR_INVALID_ARG, "a parameter-gradient array is NULL");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  const luna::Dt dt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int M = p->M, L = p->L, D = M * L, dd = (int)d, E = dd + 1;
  const int heads = (int)(B * H), C = lay.chunk, nch = lay.nch;
  const int64_t nD = n * D, nE = n * E, st_el = (int64_t)D * E, cc = (int64_t)C * C;
  float* phiq = reinterpret_cast<float*>(w + lay.phiq);
  float* phik = reinterpret_cast<float*>(w + lay.phik);
  float* vx = reinterpret_cast<float*>(w + lay.vx);
  float* y = reinterpret_cast<float*>(w + lay.y);
  float* sx = reinterpret_cast<float*>(w + lay.sx);
  float* dsx = reinterpret_cast<float*>(w + lay.dsx);
  float* pm = reinterpret_cast<float*>(w + lay.pm);
  float* rm = reinterpret_cast<float*>(w + lay.rm);
  float* dphiq = reinterpret_cast<float*>(w + lay.dphiq);
  float* dphik = reinterpret_cast<float*>(w + lay.dphik);
  float* dvf = dt == luna::Dt::BF16 ? reinterpret_cast<float*>(w + lay.dvtmp) : static_cast<float*>(dV);
  hipError_t e;
#define LUNA_TRY(expr, what) \
  if ((e = (expr)) != hipSuccess) return hip_fail(e, what)
  // the forward pass in fp32: features, [V | 1], states, [num | den - eps] (and P)
  if ((st = enqueue_f32_forward(pb, w, lay, Q, K, V, causal != 0, s)) != LUNA_OK) return st;
  const ChunkGemm gemm{heads, nch, C, (int)n, s};
  const int64_t sh = (int64_t)nch * st_el;  // head stride of the per-chunk states
  LUNA_TRY(luna::launch_bwd_g(dt, y, dO, (int64_t)heads * n, dd, eps, s), "denominator kernel launch");
  // dphi(Q_c) = G_c [S_c | z_c]^T (+ R_c phi(K_c), R_c = tril(G_c [V_c | 1]^T))
  LUNA_TRY(gemm(y, nE, (int64_t)C * E, E, 1, sx, sh, st_el, 1, E, dphiq, nD, (int64_t)C * D, D, 1, C, D, E, 1, 0, 0,
                0, 0), "dphi(Q) GEMM");
  if (causal) {
    LUNA_TRY(gemm(y, nE, (int64_t)C * E, E, 1, vx, nE, (int64_t)C * E, 1, E, rm, nch * cc, cc, C, 1, C, C, E, 1, 1, 0,
                  1, 0), "R GEMM");
    LUNA_TRY(gemm(rm, nch * cc, cc, C, 1, phik, nD, (int64_t)C * D, D, 1, dphiq, nD, (int64_t)C * D, D, 1, C, D, C, 1,
                  0, 1, 0, 1), "dphi(Q) intra-chunk GEMM");
  }
  // per-chunk [dS | dz] = phi(Q_c)^T G_c, then exclusive suffix over chunks (causal)
  LUNA_TRY(gemm(phiq, nD, (int64_t)C * D, 1, D, y, nE, (int64_t)C * E, E, 1, dsx, sh, st_el, E, 1, D, E, C, 0, 0, 1,
                0, 0), "state-gradient GEMM");
  LUNA_TRY(luna::launch_bwd_scan(dsx, heads, nch, st_el, causal ? 1 : 2, s), "state-gradient scan");
  // dphi(K_c) = [V_c | 1] [dS_c | dz_c]^T (+ R_c^T phi(Q_c)); dV_c = phi(K_c) dS_c (+ P_c^T dnum_c)
  LUNA_TRY(gemm(vx, nE, (int64_t)C * E, E, 1, dsx, sh, st_el, 1, E, dphik, nD, (int64_t)C * D, D, 1, C, D, E, 1, 0, 0,
                0, 0), "dphi(K) GEMM");
  LUNA_TRY(gemm(phik, nD, (int64_t)C * D, D, 1, dsx, sh, st_el, E, 1, dvf, n * dd, (int64_t)C * dd, dd, 1, C, dd, D, 1,
                0, 0, 0, 0), "dV GEMM");
  if (causal) {
    LUNA_TRY(gemm(rm, nch * cc, cc, 1, C, phiq, nD, (int64_t)C * D, D, 1, dphik, nD, (int64_t)C * D, D, 1, C, D, C, 1,
                  0, 1, 0, 1), "dphi(K) intra-chunk GEMM");
    LUNA_TRY(gemm(pm, nch * cc, cc, 1, C, y, nE, (int64_t)C * E, E, 1, dvf, n * dd, (int64_t)C * dd, dd, 1, C, dd, C, 1,
                  0, 1, 0, 1), "dV intra-chunk GEMM");
  }
  if (dt == luna::Dt::BF16) LUNA_TRY(luna::launch_bwd_convert(dt, dvf, dV, (int64_t)heads * n * dd, s), "dV convert");
  return enqueue_phi_backward(pb, w, lay, Q, K, dQ, dK, grads, s);
#undef LUNA_TRY
}

size_t luna_distill_workspace_bytes(luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                                    const luna_phi_params* p, int32_t param_grads) {
  Problem pb{param_grads ? kOpDistillGrads : kOpDistill, dtype, B, H, n, d, p, 64};
  Layout lay;
  return plan(pb, &lay) == LUNA_OK ? lay.total : 0;
}

luna_status luna_distill(const void* Q, const void* K, luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                         const luna_phi_params* p, int32_t causal, float eps, float* row_loss,
                         const luna_phi_grads* grads, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (causal != 0 && causal != 1) return fail(LUNA_ERR_INVALID_ARG, "causal must be 0 or 1");
  Problem pb{grads ? kOpDistillGrads : kOpDistill, dtype, B, H, n, d, p, 64};
  Layout lay;
  luna_status st = plan(pb, &lay);
  if (st != LUNA_OK) return st;
  if (!Q || !K || !row_loss) return fail(LUNA_ERR_INVALID_ARG, "Q, K or row_loss is NULL");
  if (grads && (!grads->W || !grads->b || !grads->fc1_w || !grads->fc1_b || !grads->fc2_w || !grads->fc2_b))
    return fail(LUNA_ERR_INVALID_ARG, "a parameter-gradient array is NULL");
  if (!finite_nonneg(eps)) return fail(LUNA_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (B * H * ((n + 63) / 64) > ((int64_t)1 << 31) - 1) return fail(LUNA_ERR_UNSUPPORTED, "too many 64-row tiles");
  if ((st = check_ws(lay, ws, ws_bytes)) != LUNA_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = static_cast<uint8_t*>(ws);
  if ((st = enqueue_prepare(pb, w, lay, s)) != LUNA_OK) return st;
  const luna::Dt dt = dtype == LUNA_BF16 ? luna::Dt::BF16 : luna::Dt::F32;
  const int D = p->M * p->L;
  luna::FeatureMapArgs f{};  // features of the queries and keys in the call's dtype, one launch
  f.phi = phi_args(pb, w, lay);
  f.rows_per_head = n;
  f.H = (int)H;
  f.heads = B * H;
  f.X = K;
  f.out = w + lay.phik;
  f.X2 = Q;
  f.out2 = w + lay.phiq;
  hipError_t e = luna::launch_featuremap(dt, dt, (int)d, p->L, f, s);
  if (e != hipSuccess) return hip_fail(e, "feature-map kernel launch");
  luna::DistillArgs a{};
  a.Q = Q;
  a.K = K;
  a.phiq = w + lay.phiq;
  a.phik = w + lay.phik;
  a.stats = reinterpret_cast<float*>(w + lay.dstats);
  a.row_loss = row_loss;
  a.dphiq = grads ? reinterpret_cast<float*>(w + lay.dphiq) : nullptr;
  a.dphik = grads ? reinterpret_cast<float*>(w + lay.dphik) : nullptr;
  a.n = n;
  a.heads = B * H;
  a.causal = causal;
  a.scale = 1.0f / std::sqrt((float)d);
  a.eps = eps;
  a.inv_rows = (float)(1.0 / ((double)B * (double)H * (double)n));
  if ((e = luna::launch_distill(dt, (int)d, D, a, grads != nullptr, s)) != hipSuccess)
    return hip_fail(e, "distillation kernel launch");
  if (!grads) return LUNA_OK;
  return enqueue_phi_backward(pb, w, lay, Q, K, nullptr, nullptr, grads, s);
}

const char* luna_status_string(luna_status s) {
  switch (s) {
    case LUNA_OK: return "ok";
    case LUNA_ERR_INVALID_ARG: return "invalid argument";
    case LUNA_ERR_UNSUPPORTED: return "unsupported problem";
    case LUNA_ERR_WORKSPACE: return "workspace too small";
    case LUNA_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* luna_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
