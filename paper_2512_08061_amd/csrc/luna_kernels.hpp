// luna_kernels.hpp -- interface between the host API (luna_api.cpp) and the kernels.
// Internal: not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace luna {

// piecewise-linear tables of the channel MLPs (built by luna_prepare.hip)
//
// Layout of one table (kTableBytes, a multiple of 256):
//   header   PwlHeader
//   keys     the sorted breakpoints, fp32, padded with +inf to PwlHeader::nkeys
//            (one window past the last breakpoint when that fits)
//   buckets  uint16 per bucket of u: byte offset (4 * index) of its search window
//   segments (slope, intercept) pairs, segment-major, L per segment, fp32:
//            psi_l(u) = slope u + intercept on the segment
//   segments16 rows of seg16_row_bytes(L) bytes for the bf16 attention paths: per
//            channel an fp16 pair (slope, value at the anchor), then the segment's
//            anchor a (fp32): psi_l(u) = slope (u - a) + value.  The anchor is the
//            segment's left breakpoint (the first segment's right one; 0 without
//            breakpoints), so |u - a| stays within the segment and the fp16 rounding
//            of slope and value is relative to the channel's size there, not to an
//            intercept that cancels against slope u.  Slopes and values are scaled by
//            2^scale_exp (the largest magnitude lands near 2^14), which cancels between
//            numerator and denominator once eps is scaled alike.
//   first    fp32 per bucket: the key its first halving compares against (the one at
//            index start + 2^(steps - 1) - 1 of its window; 0 when steps = 0), so that
//            a search can read it together with the window start
//
// Search.  The float bits of u pick one of kNumBuckets buckets (bucket_of), an
// order-preserving partition of the real line: sign, then |u| below 2^-kBucketExp,
// in [2^-kBucketExp, 2^kBucketExp) split by exponent and the top kBucketMant
// mantissa bits, or above.  Every breakpoint that can lie below a u of the bucket,
// beyond those below the whole bucket, sits inside a window of 2^steps - 1 keys
// starting at the bucket's offset, so `steps` branch-free halvings of the window
// give the number of breakpoints strictly below u, which is the segment index.
constexpr int kKeyCap = 1024;           // sorted breakpoints incl. +inf padding
constexpr int kSegCap = 5120;           // (slope, intercept) pairs, segment-major
constexpr int kMaxUnits = kKeyCap - 1;  // breakpoints one table can hold
constexpr int kBucketExp = 6;           // resolved magnitudes: [2^-6, 2^6)
constexpr int kBucketMant = 7;          // mantissa bits per exponent
constexpr int kBucketMag = 2 * kBucketExp * (1 << kBucketMant) + 2;  // per sign, incl. under/overflow
constexpr int kNumBuckets = 2 * kBucketMag;                          // 3076
constexpr size_t kTabHeader = 0;
constexpr size_t kTabKeys = 256;
constexpr size_t kTabBuckets = kTabKeys + kKeyCap * 4;
constexpr size_t kTabSeg = kTabBuckets + ((size_t)kNumBuckets * 2 + 15) / 16 * 16;
constexpr size_t kTabSeg16 = kTabSeg + (size_t)kSegCap * 8;
constexpr size_t kSeg16Bytes = 40960;  // fp16 rows with anchors
constexpr size_t kTabFirst = kTabSeg16 + kSeg16Bytes;
constexpr size_t kFirstBytes = ((size_t)kNumBuckets * 4 + 15) / 16 * 16;
constexpr size_t kTableBytes = (kTabFirst + kFirstBytes + 255) / 256 * 256;

struct PwlHeader {
  int nbp;     // number of breakpoints
  int steps;   // halvings per search: smallest s with 2^s - 1 >= the most keys one bucket can need
  int L;       // channels
  int nonneg;  // 1: relu on the channel outputs
  int nkeys;   // keys stored (breakpoints plus +inf padding), >= 2^steps - 1
  int scale_exp;  // fp16 slopes and values are 2^scale_exp times the fp32 ones
  int nodes;   // 1 or 2: the keys a u compares against are the first 4 or 8 from its
               // bucket's offset (no window was shifted to fit); 0 otherwise
};

// Bucket of u from its float bits; monotone in u (-0.0 and +0.0 fall in the two
// buckets next to zero, NaN in an outermost one).
__host__ __device__ constexpr int bucket_of_bits(uint32_t bits) {
  const int mag = (int)((bits >> (23 - kBucketMant)) & ((1u << (31 - 23 + kBucketMant)) - 1u));
  int m = mag - ((127 - kBucketExp) << kBucketMant) + 1;  // 0: underflow, 1..: resolved, last: overflow
  m = m < 0 ? 0 : (m > kBucketMag - 1 ? kBucketMag - 1 : m);
  return (bits >> 31) ? kBucketMag - 1 - m : kBucketMag + m;
}

enum class Dt : int { F32 = 0, BF16 = 1 };

// Build the piecewise-linear tables of the channel MLPs (one per parameter set).
struct PrepareArgs {
  const float* fc1_w;  // [P][C1][hidden]
  const float* fc1_b;  // [P][C1][hidden]
  const float* fc2_w;  // [P][L][hidden]
  const float* fc2_b;  // [P][L]
  int P, C1, L, hidden, M, nonneg;
  uint8_t* tables;     // [P][kTableBytes]
};

// Projection and channel-MLP parameters as the kernels see them.
struct PhiArgs {
  const void* W;        // [P][M][d], element type of the call
  const float* b;       // [P][M]
  const uint8_t* tables;
  int M;
  int per_head;         // parameter set = per_head ? h : 0
};

struct FeatureMapArgs {
  const void* X;
  void* out;
  const void* X2;  // non-null: a second input of the same shape, mapped into out2
  void* out2;
  PhiArgs phi;
  int64_t rows_per_head;  // n
  int H;
  int64_t heads;          // B * H
  // optional copy of copy_n floats from copy_src to copy_dst, done by workgroups of
  // the same launch beside the mapping ones (the streaming step's z before the step)
  const float* copy_src;
  float* copy_dst;
  int64_t copy_n;
  int map_grid;           // workgroups that map rows (set by the launcher)
};

struct NoncausalArgs {
  const void* Q;
  const void* K;
  const void* V;
  void* out;
  PhiArgs phi;
  int n, H, heads;
  int splits;           // token ranges per head in the state pass
  int tokens_per_split; // multiple of 32
  float eps;
  float* partial;       // [heads][splits][DP][DH + 1] fp32
  void* frags;          // [heads][frag_elems] statistics as readout fragments (call dtype)
  int tile_tokens;      // tokens per readout workgroup (multiple of 16)
  int tiles;            // ceil(n / tile_tokens)
  int fused;            // 1: one workgroup per head does state and readout
  // state export (luna_attn_state): S [heads][M*L][d] and z [heads][M*L], fp32,
  // feature i*L + l; accumulate 1 adds to them instead of overwriting
  float* state_S;
  float* state_z;
  int accumulate;
};

// Heads from which the non-causal path uses one fused workgroup per head, and the
// largest per-wave (S | z) accumulator set (fp32 registers per lane) it holds.
constexpr int kFusedMinHeads = 192;
constexpr int kFusedMaxAccRegs = 128;
__host__ __device__ constexpr int fused_acc_regs(int d, int L, int M) { return ((M + 15) / 16) * L * (d / 16) * 4; }

struct CausalArgs {
  const void* Q;
  const void* K;
  const void* V;
  void* out;
  PhiArgs phi;
  int n, H, heads;
  int parts;     // workgroups per head (1 or 2)
  int split;     // with 2 parts: first token of part 1 (a multiple of 64)
  float eps;
  // State of the first `split` tokens of every head, built beforehand in `pieces`
  // pieces of `piece_chunks` chunks each, one workgroup per (head, piece): the state
  // launch writes state_out, the scan launch's part 1 starts from the sum of the
  // pieces in state_in (causal_state_floats() floats per piece, the kernel's own layout).
  float* state_out;      // non-null: state launch
  const float* state_in;  // non-null: part 1 of the scan launch starts from the pieces
  int pieces, piece_chunks;
  // Staged scan (staged = 1, two launches of the scan kernel): part p of a launch covers
  // chunks [pc_first[p], pc_end[p]), of which [pc_first[p], pc_begin[p]) only build the
  // state; it starts from the sum of the first pseed[p] pieces of state_in (`pieces`
  // pieces per head) and, with state_fin non-null, writes its final state (S and z,
  // fp32, the pieces' layout) as piece p of its head in state_fin.
  int staged;
  int pc_first[2], pc_begin[2], pc_end[2], pseed[2];
  float* state_fin;
  // non-null: sum the pieces in state_out into S [heads][M*L][d] and z [heads][M*L]
  // (fp32, feature i*L + l; accumulate 1 adds to them) instead of launching the kernel
  float* export_S;
  float* export_z;
  int accumulate;
  // features given (launch_causal_given): phi(Q), phi(K) [heads][n][D] in bf16
  const void* phiq;
  const void* phik;
};

// One streaming step of causal attention over m new tokens per head, from the
// features of the new queries and keys (fp32, feature i*L + l) and the state (S, z),
// which is updated in place.
struct StepArgs {
  const float* phiq;  // [heads][m][D]
  const float* phik;  // [heads][m][D]
  const void* V;      // [heads][m][d], element type of the call
  void* out;          // [heads][m][d]
  float* S;           // [heads][D][d]
  float* z;           // [heads][D], written by the column block 0 of each head
  const float* z_in;  // [heads][D], z as it was before the call: every column block of a
                      // head reads this copy, never z, which block 0 overwrites
  int m, d, D, heads;
  float eps;
};
constexpr int kStepMaxD = 256;  // features the step kernel holds per column

// Backward pass (luna_backward.hip).  Batched C (+)= A B over (head, chunk) with
// strided fp32 operands: element (i, k) of A at A + h sAh + c sAc + i sAi + k sAk, and
// so on.  Dimensions marked *_chunk are token dimensions of a chunk of `chunk`
// tokens of a `seq`-token sequence (shorter in a ragged last chunk).  lower: entries
// above the diagonal (j > i) of the product are stored as 0.
struct BwdGemm {
  const float* A;
  const float* B;
  float* C;
  int M, N, K;
  int64_t sAh, sAc, sAi, sAk;
  int64_t sBh, sBc, sBk, sBj;
  int64_t sCh, sCc, sCi, sCj;
  int heads, chunks, chunk, seq;
  int m_chunk, n_chunk, k_chunk;
  int lower, accumulate;
};

// Feature-map backward over the rows of Q and K of every head, one thread per
// (row, projection): du from dphi and u, and the (segment, channel) moments.
struct BwdPhi {
  const float* uq;     // [heads][n][M] projections u = x W^T + b
  const float* uk;
  const float* dphiq;  // [heads][n][M*L]
  const float* dphik;
  float* duq;          // [heads][n][M]
  float* duk;
  const uint8_t* tables;
  float* partial;      // [P][groups][part_floats]: (segment, channel) moments
  int64_t n, heads;
  int H, M, per_head;
  int part_floats;
};

// Channel-MLP parameter gradients from the reduced partials.
struct BwdMlp {
  const double* sum;   // [P][part_floats] (fp64)
  const double* pre;   // [P][L][nseg_cap + 1][2]: exclusive prefix sums of the moments
  const uint8_t* tables;
  const float* fc1_w;
  const float* fc1_b;
  const float* fc2_w;
  float* dfc1_w;
  float* dfc1_b;
  float* dfc2_w;
  float* dfc2_b;
  int L, hidden, C1, part_floats, nseg_cap;
};

bool bwd_supported(int d, int L, int M);
size_t bwd_part_floats(int d, int L, int M);
int bwd_phi_groups(int64_t rows_per_set);
int bwd_nseg_cap(int L);
hipError_t launch_bwd_pack(Dt dt, const void* V, float* Vx, int64_t rows, int d, hipStream_t s);
hipError_t launch_bwd_convert(Dt dt, const float* src, void* dst, int64_t n, hipStream_t s);
hipError_t launch_bwd_gemm(const BwdGemm& g, hipStream_t s);
hipError_t launch_bwd_scan(float* X, int heads, int chunks, int64_t elems, int mode, hipStream_t s);
hipError_t launch_bwd_g(Dt dt, float* Y, const void* dO, int64_t rows, int d, float eps, hipStream_t s);
hipError_t launch_bwd_packw(Dt dt, const void* W, const float* b, float* Wx, int rows, int d, hipStream_t s);
hipError_t launch_bwd_phi(int L, const BwdPhi& a, int groups, int sets, hipStream_t s);
hipError_t launch_bwd_dw(const float* dwh, float* dW, float* db, int B, int H, int M, int d, int per_head,
                         hipStream_t s);
hipError_t launch_bwd_cols(Dt dt, const float* src, void* dst, int64_t rows, int d, hipStream_t s);
hipError_t launch_bwd_reduce(const float* partial, double* sum, int groups, int part_floats, int used, int sets,
                             hipStream_t s);
hipError_t launch_bwd_prefix(const double* sum, double* pre, const uint8_t* tables, int M, int d, int L,
                             int part_floats, int nseg_cap, int sets, hipStream_t s);
hipError_t launch_bwd_mlp(const BwdMlp& a, int sets, hipStream_t s);
// Feature-map variants (random Fourier cos and sin/cos, Performer, channel MLPs with a
// smooth activation, an envelope, channel RMS and Bank+Coef), evaluated directly.
constexpr int kVarMlp = 0, kVarCos = 1, kVarSinCos = 2, kVarPerformer = 3;
constexpr int kVariantMaxGrid = 2048;   // workgroups of one variant map (rows loop)
constexpr int kVariantMaxL = 16;        // channel RMS partials per workgroup
struct VariantArgs {
  const void* X;        // [heads][n][d], the call's input dtype
  void* out;            // [heads][n][D]
  const void* W;        // [P][M][d], input dtype
  const float* b;       // [P][M]
  const float* fc1_w;   // [P][C1][hidden]
  const float* fc1_b;
  const float* fc2_w;   // [P][L][hidden]
  const float* fc2_b;   // [P][L]
  const float* env_w;   // [P][L][d] or null
  const float* env_b;   // [P][L]
  const float* bank;    // [P][L] or null
  int kind, act, M, L, hidden, C1, nonneg, per_head, H;
  int64_t rows_per_head, heads;
  int out_bf16;             // phi stored as bf16 (else fp32)
  int rms_pass;             // 1: y into rms_y and sums of y^2 into rms_partial, no phi; 0: phi
  double* rms_partial;      // [grid][kVariantMaxL]
  float* rms_y;             // [heads][n][M][L]: y after the envelope, before the channel scales
};
// Launch the variant map (a.out_bf16 set); *grid receives the workgroup count, the
// number of channel-RMS partials written by a first pass.
hipError_t launch_variant_map(Dt in_dt, int d, const VariantArgs& a, int* grid, hipStream_t s);
// phi from rms_y: channel scales, bank sum or 1/sqrt(M), in the output dtype
hipError_t launch_variant_finish(const VariantArgs& a, const float* scale, hipStream_t s);
hipError_t launch_variant_rms(const double* partial, int groups, int L, double count, float target, float* scale,
                              hipStream_t s);
hipError_t launch_widen(Dt dt, const void* src, float* dst, int64_t n, hipStream_t s);

// Attention distillation (luna_distill.hip): per query row the soft cross-entropy of
// the softmax teacher against LUNA's smoothed weights, and the gradients of its mean
// with respect to the features.  Features are in the call's dtype, [head][n][D].
struct DistillArgs {
  const void* Q;       // [heads][n][d]
  const void* K;
  const void* phiq;    // [heads][n][D]
  const void* phik;
  float* stats;        // [heads][n][4]: base-2 softmax maximum, sum, den (written, then read)
  float* row_loss;     // [heads][n]
  float* dphiq;        // [heads][n][D] fp32 (gradients only)
  float* dphik;
  int64_t n, heads;
  int causal;
  float scale;         // 1 / sqrt(d)
  float eps;
  float inv_rows;      // 1 / (heads n): the gradients are of the mean
};
bool distill_supported(Dt dt, int d, int D);
hipError_t launch_distill(Dt dt, int d, int D, const DistillArgs& a, bool grads, hipStream_t s);

// forward pass of the shapes without a fused kernel (fp32 GEMMs and scans as above)
hipError_t launch_fwd_out(Dt dt, const float* Y, void* out, int64_t rows, int d, float eps, hipStream_t s);
hipError_t launch_fwd_export(const float* X, int64_t head_stride, float* S, float* z, int heads, int D, int d,
                             int accumulate, hipStream_t s);

// Launchers; each returns hipSuccess or the launch error.  `ok` reports whether
// a kernel exists for the (dtype, d, L, M) combination.
hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s);

bool featuremap_supported(Dt dt, int d, int L, int M);
hipError_t launch_featuremap(Dt in_dt, Dt out_dt, int d, int L, const FeatureMapArgs& a, hipStream_t s);

struct NoncausalPlan {
  int DP;          // padded feature rows of S (16 * MB * L)
  int NF;          // readout fragments along the feature dimension
  size_t frag_elems;  // per-head elements of the statistics fragments
};
bool noncausal_supported(Dt dt, int d, int L, int M, NoncausalPlan* plan);
hipError_t launch_noncausal(Dt dt, int d, int L, int M, const NoncausalArgs& a, hipStream_t s);
// the state pass of the non-causal split path, then its partials summed into
// state_S / state_z
hipError_t launch_state(Dt dt, int d, int L, int M, const NoncausalArgs& a, hipStream_t s);

hipError_t launch_causal_step(Dt dt, const StepArgs& a, hipStream_t s);

bool causal_supported(Dt dt, int d, int L, int M);
// floats of one state piece (S slices of the matrix waves, then z) for a combination
size_t causal_state_floats(Dt dt, int d, int L, int M);
hipError_t launch_causal(Dt dt, int d, int L, int M, const CausalArgs& a, hipStream_t s);
// The causal kernel with the features given in bf16 (D of them per token), for the
// feature maps whose projections and tables the fused kernel cannot hold.
bool causal_given_supported(Dt dt, int d, int D);
size_t causal_given_state_floats(int d, int D);
hipError_t launch_causal_given(int d, int D, const CausalArgs& a, hipStream_t s);

// LDS copy of the segment table: one row of (slope, intercept) pairs per segment.
// Rows whose size is a multiple of 64 bytes are padded by 16 bytes so that random
// segments spread over all LDS banks.
constexpr int seg_row(int L) { return (L % 8 == 0) ? L + 2 : L; }
// fp16 segment rows: L (slope, value) half2 pairs and the fp32 anchor, in whole
// 16-byte chunks, padded by 16 more bytes when that is a multiple of 64 (so that
// random rows spread over all LDS banks); the same bytes in global memory and LDS
constexpr int seg16_row_bytes(int L) {
  return ((4 * L + 4 + 15) / 16 * 16) % 64 == 0 ? (4 * L + 4 + 15) / 16 * 16 + 16 : (4 * L + 4 + 15) / 16 * 16;
}
// Segments an LDS table of `bytes` holds for L channels (at most 64 L + 2: width-64
// per-channel MLPs plus the all-zero segment).  A table needs breakpoints + 2.
constexpr int nseg_cap(int L, int bytes) {
  return (64 * L + 2) < bytes / (seg_row(L) * 8) ? (64 * L + 2) : bytes / (seg_row(L) * 8);
}
constexpr int kAttnSegBytes = 41120;  // attention kernels (514 segments at L = 8)
constexpr int kFmSegBytes = 46080;    // feature-map kernel

}  // namespace luna
