// luna_device.hpp -- device building blocks shared by the LUNA kernels (gfx950).
//
// Matrix-core fragments.  Every product in this library is built from one
// abstraction: a 16x16 output block accumulated in fp32 from operands that each
// hold, per lane, 8 values of the reduction ("k") dimension:
//
//   lane l (0..63), group g = l / 16, index r = l % 16
//   A operand: row r,    k-slots (g, e), e = 0..7
//   B operand: column r, k-slots (g, e), e = 0..7
//   C/D:       rows 4g + j (j = 0..3), column r
//
// The hardware pairs A's slot (g, e) with B's slot (g, e); which abstract k a
// slot stands for is chosen by each kernel (the same choice on both operands),
// so kernels are free to permute k to match the layout their data arrives in.
// bf16 uses one v_mfma_f32_16x16x32_bf16 per fragment pair; fp32 uses eight
// v_mfma_f32_16x16x4_f32 (instruction e consumes slot e of every group).
//
// Channel functions.  A ReLU MLP of a scalar is continuous and piecewise linear
// in that scalar.  Its breakpoints -c_k/a_k are merged and sorted once per call
// (luna_prepare.hip); evaluation is then a lookup of u's bucket (an order-preserving
// partition of the reals by float bits), which gives the start of a short window of
// sorted keys, a count of the window's keys below u (branch-free halvings, or one or
// two 16-byte reads of 4-key groups), and one fused multiply-add per channel: slope
// u + intercept (fp32 rows) or slope (u - anchor) + value at the anchor (fp16 rows of
// the bf16 paths).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "luna_kernels.hpp"

namespace luna {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(2))) int i32x2;

constexpr int kWave = 64;

// Index of the calling wave within its workgroup, as a scalar (SGPR) value.
// Matrix-core instructions execute for all 64 lanes whatever the EXEC mask is, so
// every branch that guards one must be taken by the whole wave.  Deriving the wave
// index through readfirstlane makes the compiler see it as uniform and emit scalar
// branches instead of EXEC-masked ones; all wave-dependent control flow in these
// kernels goes through this value.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

// ---------------------------------------------------------------------------
// piecewise-linear tables (layout shared with the host and luna_prepare.hip)
// ---------------------------------------------------------------------------

// Header fields as the kernels use them, clamped to what an LDS table of NSEG rows
// can hold.  The tables are built on the device at the start of a call (or, for
// streaming steps, by an earlier call on the same workspace); a workspace that never
// held them gives wrong results but no LDS access out of range and no unbounded
// search loop.
struct PwlDims {
  int nseg;   // real segments (breakpoints + 1); the all-zero segment follows them
  int steps;  // halvings per search, <= 10 (windows of at most kKeyCap - 1 keys)
  int nkeys;  // stored keys, <= kKeyCap
  int nodes;  // 0, 1 or 2 (PwlHeader::nodes)
};
template <int NSEG>
__device__ __forceinline__ PwlDims pwl_dims(const PwlHeader& hd) {
  PwlDims r;
  r.nseg = min(max(hd.nbp, 0), NSEG - 2) + 1;
  r.steps = min(max(hd.steps, 0), 10);
  r.nkeys = min(max(hd.nkeys, 0), kKeyCap);
  r.nodes = (hd.nodes == 1 || hd.nodes == 2) ? hd.nodes : 0;
  return r;
}

// LDS copy of one table for L channels, NSEG segment rows (see seg_row).
template <int L, int NSEG>
struct alignas(16) PwlLds {
  static constexpr int SROW = seg_row(L);
  float keys[kKeyCap];
  uint16_t buckets[(kNumBuckets + 7) / 8 * 8];
  float2 seg[NSEG][SROW];
  int steps;
  int zero_seg;   // index of the all-zero segment (nbp + 1)
  float floor;    // 0 when outputs are clamped at zero, -inf otherwise
  int scale_exp;  // 0: these are the unscaled values
};

// Cooperative 16-byte copies global -> LDS: `n16` chunks.
// Each thread issues up to kCopyBatch loads before it stores them, so that a copy
// costs about one memory round trip rather than one per chunk it moves.  The loads
// are unconditional (indices clamped to the last chunk): conditional ones would make
// the compiler keep the batch in scratch memory.
constexpr int kCopyBatch = 8;
__device__ inline void copy16(void* dst, const void* src, int n16) {
  uint4* d = reinterpret_cast<uint4*>(dst);
  const uint4* sp = reinterpret_cast<const uint4*>(src);
  const int nt = blockDim.x;
  for (int base = threadIdx.x; base < n16; base += kCopyBatch * nt) {
    uint4 v[kCopyBatch];
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u) v[u] = sp[min(base + u * nt, n16 - 1)];
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u)
      if (base + u * nt < n16) d[base + u * nt] = v[u];
  }
}
// One round of loads for n16 16-byte chunks: every thread issues all its loads
// (kTabBatch per round, indices clamped so that none is conditional) before it stores
// any.  ld(i) reads chunk i, st(i, v) writes it.
constexpr int kTabBatch = 16;
template <typename LD, typename ST>
__device__ inline void batched_copy(int n16, LD ld, ST st) {
  const int nt = blockDim.x;
  for (int base = threadIdx.x; base < n16; base += kTabBatch * nt) {
    uint4 v[kTabBatch];
#pragma unroll
    for (int u = 0; u < kTabBatch; ++u) v[u] = ld(min(base + u * nt, n16 - 1));
#pragma unroll
    for (int u = 0; u < kTabBatch; ++u)
      if (base + u * nt < n16) st(base + u * nt, v[u]);
  }
}

// The bucket windows and NROWS coefficient rows (SRC16 chunks each in global memory,
// DST16 in LDS) of a table, plus PRE leading chunks of keys, in one round of loads.
// The loads cover the capacities, not the table's own counts, so that none waits for
// the header; only the first rows_kept rows are stored (the caller writes the row
// after them).
template <int PRE, int NROWS, int SRC16, int DST16>
__device__ inline void copy_table_regions(void* keys_dst, void* bk_dst, void* seg_dst, const uint8_t* gtab,
                                          size_t seg_off, int rows_kept) {
  constexpr int NB = (kNumBuckets * 2 + 15) / 16;
  const uint4* gk = reinterpret_cast<const uint4*>(gtab + kTabKeys);
  const uint4* gb = reinterpret_cast<const uint4*>(gtab + kTabBuckets);
  const uint4* gs = reinterpret_cast<const uint4*>(gtab + seg_off);
  uint4* kd = reinterpret_cast<uint4*>(keys_dst);
  uint4* bd = reinterpret_cast<uint4*>(bk_dst);
  uint4* sd = reinterpret_cast<uint4*>(seg_dst);
  batched_copy(
      PRE + NB + NROWS * SRC16,
      [&](int i) { return i < PRE ? gk[i] : (i < PRE + NB ? gb[i - PRE] : gs[i - PRE - NB]); },
      [&](int i, uint4 v) {
        if (i < PRE) {
          kd[i] = v;
        } else if (i < PRE + NB) {
          bd[i - PRE] = v;
        } else {
          const int j = i - PRE - NB;
          if (j / SRC16 < rows_kept) sd[(j / SRC16) * DST16 + j % SRC16] = v;  // (the rest may be written after)
        }
      });
}

// Cooperative copy of a table from global memory into LDS.  Caller syncs after.
template <int L, int NSEG>
__device__ inline void pwl_load(PwlLds<L, NSEG>& t, const uint8_t* __restrict__ gtab) {
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(gtab + kTabHeader);
  const PwlDims dm = pwl_dims<NSEG>(hd);
  const int nseg = dm.nseg;
  const float* gkeys = reinterpret_cast<const float*>(gtab + kTabKeys);
  const uint32_t* gbk = reinterpret_cast<const uint32_t*>(gtab + kTabBuckets);
  const float2* gseg = reinterpret_cast<const float2*>(gtab + kTabSeg);
  static_assert(NSEG * L <= kSegCap, "the LDS rows must lie inside the table's segment region");
  if constexpr ((L * 8) % 16 == 0) {
    copy_table_regions<kKeyCap / 4, NSEG, L * 8 / 16, sizeof(t.seg[0]) / 16>(t.keys, t.buckets, &t.seg[0][0], gtab,
                                                                             kTabSeg, nseg);
  } else {
    copy16(t.keys, gkeys, (dm.nkeys + 3) / 4);
    copy16(t.buckets, gbk, (kNumBuckets * 2 + 15) / 16);
    for (int i = threadIdx.x; i < nseg * L; i += blockDim.x) t.seg[i / L][i % L] = gseg[i];
  }
  // one all-zero segment after the real ones: masked values select it and evaluate
  // to exactly 0 without per-element masks
  for (int i = threadIdx.x; i < L; i += blockDim.x) t.seg[nseg][i] = make_float2(0.0f, 0.0f);
  if (threadIdx.x == 0) {
    t.steps = dm.steps;
    t.zero_seg = nseg;
    t.floor = hd.nonneg ? 0.0f : -__builtin_inff();
    t.scale_exp = 0;
  }
}

// The same table with fp16 rows (bf16 attention paths): per channel the slope and
// the value at the segment's anchor, then the anchor in fp32 (seg16_row_bytes), read
// with mixed-precision fused multiply-adds: psi_l(u) = slope (u - anchor) + value.
typedef __attribute__((ext_vector_type(2))) _Float16 half2_t;
template <int L, int NSEG>
struct alignas(16) PwlLds16 {
  static constexpr int SROW = seg16_row_bytes(L) / 4;
  float keys[kKeyCap];
  uint16_t buckets[(kNumBuckets + 7) / 8 * 8];
  half2_t seg[NSEG][SROW];
  int steps;
  int zero_seg;
  float floor;
  int scale_exp;
};

template <int L, int NSEG>
__device__ inline void pwl_load(PwlLds16<L, NSEG>& t, const uint8_t* __restrict__ gtab) {
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(gtab + kTabHeader);
  const PwlDims dm = pwl_dims<NSEG>(hd);
  const int nseg = dm.nseg;
  const float* gkeys = reinterpret_cast<const float*>(gtab + kTabKeys);
  const uint32_t* gbk = reinterpret_cast<const uint32_t*>(gtab + kTabBuckets);
  constexpr int R16 = seg16_row_bytes(L) / 16;
  static_assert(sizeof(t.seg[0]) == 16 * R16, "LDS rows are the global rows");
  static_assert(NSEG * 16 * R16 <= (int)kSeg16Bytes, "the LDS rows must lie inside the table's fp16 region");
  copy_table_regions<kKeyCap / 4, NSEG, R16, R16>(t.keys, t.buckets, &t.seg[0][0], gtab, kTabSeg16, nseg);
  // the all-zero segment (its anchor 0 too, so that it evaluates to 0 for finite u)
  for (int i = threadIdx.x; i < PwlLds16<L, NSEG>::SROW; i += blockDim.x)
    t.seg[nseg][i] = half2_t{(_Float16)0.0f, (_Float16)0.0f};
  if (threadIdx.x == 0) {
    t.steps = dm.steps;
    t.zero_seg = nseg;
    t.floor = hd.nonneg ? 0.0f : -__builtin_inff();
    t.scale_exp = hd.scale_exp;
  }
}

// The fp16-row table plus every bucket's first comparison key, so that a search reads
// the key of its first halving together with its window start (one dependent LDS
// round trip fewer per lookup).
template <int L, int NSEG>
struct alignas(16) PwlLds16F : PwlLds16<L, NSEG> {
  float first[kFirstBytes / 4];
};

template <int L, int NSEG>
__device__ inline void pwl_load(PwlLds16F<L, NSEG>& t, const uint8_t* __restrict__ gtab) {
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(gtab + kTabHeader);
  const PwlDims dm = pwl_dims<NSEG>(hd);
  const int nseg = dm.nseg;
  constexpr int R16 = seg16_row_bytes(L) / 16;
  constexpr int NK = kKeyCap / 4, NB = (kNumBuckets * 2 + 15) / 16, NF = (int)(kFirstBytes / 16);
  static_assert(sizeof(t.seg[0]) == 16 * R16, "LDS rows are the global rows");
  static_assert(NSEG * 16 * R16 <= (int)kSeg16Bytes, "the LDS rows must lie inside the table's fp16 region");
  const uint4* gk = reinterpret_cast<const uint4*>(gtab + kTabKeys);
  const uint4* gb = reinterpret_cast<const uint4*>(gtab + kTabBuckets);
  const uint4* gf = reinterpret_cast<const uint4*>(gtab + kTabFirst);
  const uint4* gs = reinterpret_cast<const uint4*>(gtab + kTabSeg16);
  uint4* kd = reinterpret_cast<uint4*>(t.keys);
  uint4* bd = reinterpret_cast<uint4*>(t.buckets);
  uint4* fd = reinterpret_cast<uint4*>(t.first);
  uint4* sd = reinterpret_cast<uint4*>(&t.seg[0][0]);
  // one round of loads over all four regions (capacities, so that none waits for the header)
  batched_copy(
      NK + NB + NF + NSEG * R16,
      [&](int i) {
        return i < NK ? gk[i] : (i < NK + NB ? gb[i - NK] : (i < NK + NB + NF ? gf[i - NK - NB] : gs[i - NK - NB - NF]));
      },
      [&](int i, uint4 v) {
        if (i < NK) kd[i] = v;
        else if (i < NK + NB) bd[i - NK] = v;
        else if (i < NK + NB + NF) fd[i - NK - NB] = v;
        else if ((i - NK - NB - NF) / R16 < nseg) sd[i - NK - NB - NF] = v;
      });
  for (int i = threadIdx.x; i < PwlLds16<L, NSEG>::SROW; i += blockDim.x)
    t.seg[nseg][i] = half2_t{(_Float16)0.0f, (_Float16)0.0f};
  if (threadIdx.x == 0) {
    t.steps = dm.steps;
    t.zero_seg = nseg;
    t.floor = hd.nonneg ? 0.0f : -__builtin_inff();
    t.scale_exp = hd.scale_exp;
  }
}

// Segment row `seg` of a table (a 24-bit multiply: the 32-bit one is quarter rate).
template <typename Tab>
__device__ __forceinline__ const char* seg_ptr(const Tab& t, int seg) {
  return reinterpret_cast<const char*>(&t.seg[0][0]) + __umul24((unsigned)seg, (unsigned)sizeof(t.seg[0]));
}

// Argument of the segment's linear form: u - anchor for fp16 rows, u for fp32 rows
// (whose intercepts are at u = 0).
template <int L, int NSEG>
__device__ __forceinline__ float pwl_local(const PwlLds<L, NSEG>&, int, float u) {
  return u;
}
template <int L, int NSEG>
__device__ __forceinline__ float pwl_local(const PwlLds16<L, NSEG>& t, int seg, float u) {
  return u - *reinterpret_cast<const float*>(seg_ptr(t, seg) + 4 * L);
}

// relu that propagates NaN like Listing 1's ReLU (fmaxf would drop it); one
// v_maximum3_f32 on gfx950.
__device__ __forceinline__ float relu_floor(float v, float floor) {
  return __builtin_elementwise_maximum(v, floor);
}

// Bucket of u: its float bits' sign, then exponent and top mantissa bits over
// [2^-kBucketExp, 2^kBucketExp), clamped into the underflow and overflow buckets.
__device__ __forceinline__ int pwl_bucket(float u) {
  const uint32_t bits = __float_as_uint(u);
  const int mag = (int)((bits >> (23 - kBucketMant)) & ((1u << (31 - 23 + kBucketMant)) - 1u));
  int mm = mag - ((127 - kBucketExp) << kBucketMant) + 1;
  mm = min(max(mm, 0), kBucketMag - 1);
  return kBucketMag + (mm ^ ((int)bits >> 31));
}

// The same search, ending in the byte offset 4 seg of the segment's key instead of
// seg.  The halvings are unrolled for the usual step counts, so that every key read
// addresses `off` plus a constant that the LDS instruction's offset field carries:
// a step then costs one compare, one select and one add.
template <int STEPS, int NU, typename Tab>
__device__ __forceinline__ void pwl_halvings(const Tab& t, const float (&u)[NU], unsigned (&off)[NU]) {
  const char* keys = reinterpret_cast<const char*>(t.keys);
#pragma unroll
  for (int s = STEPS - 1; s >= 0; --s) {
    const unsigned h4 = 4u << s;
#pragma unroll
    for (int i = 0; i < NU; ++i) {
      const float key = *reinterpret_cast<const float*>(keys + off[i] + (h4 - 4u));
      off[i] += key < u[i] ? h4 : 0u;
    }
  }
}
template <int NU, typename Tab>
__device__ __forceinline__ void pwl_search_off(const Tab& t, int steps, const float (&u)[NU], unsigned (&off)[NU]) {
#pragma unroll
  for (int i = 0; i < NU; ++i) off[i] = t.buckets[pwl_bucket(u[i])];
  switch (steps) {
    case 0: break;
    case 1: pwl_halvings<1>(t, u, off); break;
    case 2: pwl_halvings<2>(t, u, off); break;
    case 3: pwl_halvings<3>(t, u, off); break;
    case 4: pwl_halvings<4>(t, u, off); break;
    default: {
      const char* keys = reinterpret_cast<const char*>(t.keys);
      for (int s = steps - 1; s >= 0; --s) {
        const unsigned h4 = 4u << s;
#pragma unroll
        for (int i = 0; i < NU; ++i) {
          const float key = *reinterpret_cast<const float*>(keys + off[i] + h4 - 4u);
          off[i] += key < u[i] ? h4 : 0u;
        }
      }
    }
  }
}

// Segment index of each of NU values: the number of breakpoints strictly below u.
// The bucket of u gives the start of its key window; `steps` halvings of the
// window follow (a wave-uniform count, taken from the table).  The NU searches
// advance together, so each step issues NU independent LDS reads and the lookup
// latency is paid once per step rather than once per value.  NaN compares false
// everywhere and ends at the start of its window.
template <int NU, typename Tab>
__device__ __forceinline__ void pwl_search(const Tab& t, int steps, const float (&u)[NU], int (&seg)[NU]) {
  // (one loop over the steps: unrolled halvings, as in pwl_search_off, measured 1-3%
  // slower in the non-causal kernel, whose code they make a fifth longer)
  const char* keys = reinterpret_cast<const char*>(t.keys);
  unsigned off[NU];
#pragma unroll
  for (int i = 0; i < NU; ++i) off[i] = t.buckets[pwl_bucket(u[i])];
  for (int s = steps - 1; s >= 0; --s) {
    const unsigned h4 = 4u << s;
#pragma unroll
    for (int i = 0; i < NU; ++i) {
      const float key = *reinterpret_cast<const float*>(keys + off[i] + h4 - 4u);
      off[i] += key < u[i] ? h4 : 0u;
    }
  }
#pragma unroll
  for (int i = 0; i < NU; ++i) seg[i] = (int)(off[i] >> 2);
}

// Segment index of each of NU values (as pwl_search) with the first halving's key read
// beside the window start.
template <int NU, typename Tab>
__device__ __forceinline__ void pwl_search_first(const Tab& t, int steps, const float (&u)[NU], int (&seg)[NU]) {
  const char* keys = reinterpret_cast<const char*>(t.keys);
  unsigned off[NU];
  float k1[NU];
#pragma unroll
  for (int i = 0; i < NU; ++i) {
    const int b = pwl_bucket(u[i]);
    off[i] = t.buckets[b];
    k1[i] = t.first[b];
  }
  if (steps > 0) {
    const unsigned h4 = 4u << (steps - 1);
#pragma unroll
    for (int i = 0; i < NU; ++i) off[i] += k1[i] < u[i] ? h4 : 0u;
  }
  for (int s = steps - 2; s >= 0; --s) {
    const unsigned h4 = 4u << s;
#pragma unroll
    for (int i = 0; i < NU; ++i) {
      const float key = *reinterpret_cast<const float*>(keys + off[i] + h4 - 4u);
      off[i] += key < u[i] ? h4 : 0u;
    }
  }
#pragma unroll
  for (int i = 0; i < NU; ++i) seg[i] = (int)(off[i] >> 2);
}
template <int NU, int L, int NSEG>
__device__ __forceinline__ void pwl_search(const PwlLds16F<L, NSEG>& t, int steps, const float (&u)[NU],
                                           int (&seg)[NU]) {
  pwl_search_first(t, steps, u, seg);
}


// psi_l(u), l = 0..L-1, on the segment whose key sits at byte offset `off` (4 seg):
// the segment row starts at off * (row bytes / 4), one multiply-add from `off`.
template <int L, int NSEG>
__device__ __forceinline__ void pwl_eval_off(const PwlLds<L, NSEG>& t, unsigned off, float floor, float u,
                                             float (&y)[L]) {
  constexpr unsigned kRow = sizeof(t.seg[0]);
  static_assert(kRow % 4 == 0 && L % 2 == 0, "rows of whole float4 pairs");
  const char* row = reinterpret_cast<const char*>(&t.seg[0][0]) + __umul24(off, kRow / 4);
#pragma unroll
  for (int q = 0; q < L / 2; ++q) {
    const float4 v = reinterpret_cast<const float4*>(row)[q];
    y[2 * q] = relu_floor(fmaf(v.x, u, v.y), floor);
    y[2 * q + 1] = relu_floor(fmaf(v.z, u, v.w), floor);
  }
}
template <int L, int NSEG>
__device__ __forceinline__ void pwl_eval_off(const PwlLds16<L, NSEG>& t, unsigned off, float floor, float u,
                                             float (&y)[L]) {
  constexpr unsigned kRow = sizeof(t.seg[0]);
  static_assert(kRow % 4 == 0 && L % 4 == 0, "rows of whole 16-byte channel quads");
  typedef __attribute__((ext_vector_type(8))) _Float16 half8_t;
  const char* row = reinterpret_cast<const char*>(&t.seg[0][0]) + __umul24(off, kRow / 4);
#pragma unroll
  for (int q = 0; q < L / 4; ++q) {
    const half8_t v = reinterpret_cast<const half8_t*>(row)[q];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      y[4 * q + i] = relu_floor(__builtin_fmaf((float)v[2 * i], u, (float)v[2 * i + 1]), floor);
  }
}

// psi_l(u) for l = 0..L-1 on segment `seg`, already scaled by 1/sqrt(M) (folded
// into the table).
template <int L, int NSEG>
__device__ __forceinline__ void pwl_channels(const PwlLds<L, NSEG>& t, int seg, float floor, float u,
                                             float (&y)[L]) {
  if constexpr (L % 2 == 0) {
    const float4* st = reinterpret_cast<const float4*>(seg_ptr(t, seg));
#pragma unroll
    for (int q = 0; q < L / 2; ++q) {
      const float4 v = st[q];
      y[2 * q] = relu_floor(fmaf(v.x, u, v.y), floor);
      y[2 * q + 1] = relu_floor(fmaf(v.z, u, v.w), floor);
    }
  } else {
#pragma unroll
    for (int l = 0; l < L; ++l) {
      const float2 v = reinterpret_cast<const float2*>(seg_ptr(t, seg))[l];
      y[l] = relu_floor(fmaf(v.x, u, v.y), floor);
    }
  }
}

// Channels 2q and 2q+1 on segment `seg` (one 16-byte LDS read).
template <int L, int NSEG>
__device__ __forceinline__ void pwl_pair(const PwlLds<L, NSEG>& t, int seg, int q, float floor, float u,
                                         float& y0, float& y1) {
  static_assert(L % 2 == 0, "channel pairs need an even L");
  const float4 v = reinterpret_cast<const float4*>(seg_ptr(t, seg))[q];
  y0 = relu_floor(fmaf(v.x, u, v.y), floor);
  y1 = relu_floor(fmaf(v.z, u, v.w), floor);
}

// fp16-row versions (slopes and values scaled by 2^scale_exp): u is the raw
// projection, the anchor is read from the row
template <int L, int NSEG>
__device__ __forceinline__ void pwl_channels(const PwlLds16<L, NSEG>& t, int seg, float floor, float u,
                                             float (&y)[L]) {
  const float x = pwl_local(t, seg, u);
  if constexpr (L % 4 == 0) {
    typedef __attribute__((ext_vector_type(8))) _Float16 half8_t;
    const half8_t* st = reinterpret_cast<const half8_t*>(seg_ptr(t, seg));
#pragma unroll
    for (int q = 0; q < L / 4; ++q) {
      const half8_t v = st[q];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        y[4 * q + i] = relu_floor(__builtin_fmaf((float)v[2 * i], x, (float)v[2 * i + 1]), floor);
    }
  } else {
#pragma unroll
    for (int l = 0; l < L; ++l) {
      const half2_t v = reinterpret_cast<const half2_t*>(seg_ptr(t, seg))[l];
      y[l] = relu_floor(__builtin_fmaf((float)v[0], x, (float)v[1]), floor);
    }
  }
}
// Channels 2q and 2q+1 from the segment's local argument x = pwl_local(t, seg, u)
// (taken once per value by the caller, which evaluates the channels pair by pair).
template <int L, int NSEG>
__device__ __forceinline__ void pwl_pair_local(const PwlLds16<L, NSEG>& t, int seg, int q, float floor, float x,
                                               float& y0, float& y1) {
  static_assert(L % 2 == 0, "channel pairs need an even L");
  typedef __attribute__((ext_vector_type(4))) _Float16 half4_t;
  const half4_t v = reinterpret_cast<const half4_t*>(seg_ptr(t, seg))[q];
  y0 = relu_floor(__builtin_fmaf((float)v[0], x, (float)v[1]), floor);
  y1 = relu_floor(__builtin_fmaf((float)v[2], x, (float)v[3]), floor);
}
template <int L, int NSEG>
__device__ __forceinline__ void pwl_pair_local(const PwlLds<L, NSEG>& t, int seg, int q, float floor, float x,
                                               float& y0, float& y1) {
  pwl_pair(t, seg, q, floor, x, y0, y1);
}

// A table whose keys are stored as overlapping groups: node s holds keys s .. s + 3
// (+inf past the stored keys), so that the keys one u compares against -- the first
// 4 or 8 from its bucket's offset when the header's `nodes` is 1 or 2 -- arrive in
// one or two aligned 16-byte loads instead of a chain of dependent halvings.  RowT
// is the coefficient pair type: half2_t (fp16, scaled) or float2.
template <typename RowT, int L, int NSEG>
struct alignas(16) PwlLdsN {
  static constexpr bool kHalf = sizeof(RowT) == 4;
  static constexpr int SROW = kHalf ? seg16_row_bytes(L) / 4 : seg_row(L);
  float4 nodes[kKeyCap + 8];
  uint16_t buckets[(kNumBuckets + 7) / 8 * 8];
  RowT seg[NSEG][SROW];
  int steps;
  int nodes_per_u;  // the header's `nodes`
  int zero_seg;     // index of the all-zero segment (nbp + 1)
  float floor;      // 0 when outputs are clamped at zero, -inf otherwise
  int scale_exp;    // fp16 rows hold 2^scale_exp times the values
};

template <typename RowT, int L, int NSEG>
__device__ inline void pwl_load(PwlLdsN<RowT, L, NSEG>& t, const uint8_t* __restrict__ gtab) {
  using Tab = PwlLdsN<RowT, L, NSEG>;
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(gtab + kTabHeader);
  const PwlDims dm = pwl_dims<NSEG>(hd);
  const int nseg = dm.nseg;
  const float* gkeys = reinterpret_cast<const float*>(gtab + kTabKeys);
  const RowT* gseg = reinterpret_cast<const RowT*>(gtab + (Tab::kHalf ? kTabSeg16 : kTabSeg));
  // groups 4m .. 4m + 3 from the aligned key quads m and m + 1 (+inf past the stored keys)
  static_assert((kKeyCap + 8) % 4 == 0, "whole quads of groups");
  const float kInf = __builtin_inff();
  constexpr int kGroups = (kKeyCap + 8) / 4;
  // this thread's first node group's key quads, loaded before the other regions'
  // round of loads so that they arrive together
  const float4* gq = reinterpret_cast<const float4*>(gkeys);
  const int m0 = threadIdx.x;
  const float4 q0 = gq[min(m0, kKeyCap / 4 - 1)], q1 = gq[min(m0 + 1, kKeyCap / 4 - 1)];
  constexpr int kPair = sizeof(RowT);
  if constexpr (Tab::kHalf) {
    constexpr int R16 = seg16_row_bytes(L) / 16;
    static_assert(sizeof(t.seg[0]) == 16 * R16, "LDS rows are the global rows");
    static_assert(NSEG * 16 * R16 <= (int)kSeg16Bytes, "the LDS rows must lie inside the table's fp16 region");
    copy_table_regions<0, NSEG, R16, R16>(nullptr, t.buckets, &t.seg[0][0], gtab, kTabSeg16, nseg);
  } else if constexpr ((L * kPair) % 16 == 0) {
    static_assert(NSEG * L <= kSegCap, "the LDS rows must lie inside the table's segment region");
    copy_table_regions<0, NSEG, L * kPair / 16, sizeof(t.seg[0]) / 16>(nullptr, t.buckets, &t.seg[0][0], gtab,
                                                                       kTabSeg, nseg);
  } else {
    copy16(t.buckets, gtab + kTabBuckets, (kNumBuckets * 2 + 15) / 16);
    for (int i = threadIdx.x; i < nseg * L; i += blockDim.x) t.seg[i / L][i % L] = gseg[i];
  }
  // groups 4m .. 4m + 3 from the aligned key quads m and m + 1 (+inf past the stored keys)
  for (int m = m0; m < kGroups; m += blockDim.x) {
    float k[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = m + h;  // key quad
      float4 v = m == m0 ? (h == 0 ? q0 : q1) : gq[min(q, kKeyCap / 4 - 1)];
      if (4 * q >= kKeyCap) v = make_float4(kInf, kInf, kInf, kInf);
      k[4 * h + 0] = v.x; k[4 * h + 1] = v.y; k[4 * h + 2] = v.z; k[4 * h + 3] = v.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (4 * m + e >= dm.nkeys) k[e] = kInf;
#pragma unroll
    for (int e = 0; e < 4; ++e) t.nodes[4 * m + e] = make_float4(k[e], k[e + 1], k[e + 2], k[e + 3]);
  }
  // one all-zero segment after the real ones (fp16 rows: its anchor 0 too): masked
  // values select it and evaluate to exactly 0 without per-element masks
  for (int i = threadIdx.x; i < Tab::SROW; i += blockDim.x) t.seg[nseg][i] = RowT{};
  if (threadIdx.x == 0) {
    t.steps = dm.steps;
    t.nodes_per_u = dm.nodes;
    t.zero_seg = nseg;
    t.floor = hd.nonneg ? 0.0f : -__builtin_inff();
    t.scale_exp = Tab::kHalf ? hd.scale_exp : 0;
  }
}

// Number of the four keys of `k` below u (NaN compares false everywhere).
__device__ __forceinline__ unsigned keys_below(const float4& k, float u) {
  return (unsigned)(k.x < u) + (unsigned)(k.y < u) + (unsigned)(k.z < u) + (unsigned)(k.w < u);
}

// Byte offset 4 seg of the segment of each u (seg = number of breakpoints below u):
// bucket offset plus the count over its one or two key groups, or, when the table
// has no node form (`nodes` 0), the halving search over node-strided keys.
template <int NU, typename RowT, int L, int NSEG>
__device__ __forceinline__ void pwl_search_n(const PwlLdsN<RowT, L, NSEG>& t, int steps, int nodes,
                                             const float (&u)[NU], unsigned (&off)[NU]) {
  const char* nb = reinterpret_cast<const char*>(t.nodes);
  unsigned s16[NU];  // byte offset of the window's first node: 16 x its first key
#pragma unroll
  for (int i = 0; i < NU; ++i) s16[i] = 4u * t.buckets[pwl_bucket(u[i])];
  if (nodes == 1) {
#pragma unroll
    for (int i = 0; i < NU; ++i)
      off[i] = (s16[i] >> 2) + 4u * keys_below(*reinterpret_cast<const float4*>(nb + s16[i]), u[i]);
  } else if (nodes == 2) {
#pragma unroll
    for (int i = 0; i < NU; ++i)
      off[i] = (s16[i] >> 2) + 4u * (keys_below(*reinterpret_cast<const float4*>(nb + s16[i]), u[i]) +
                                     keys_below(*reinterpret_cast<const float4*>(nb + s16[i] + 64), u[i]));
  } else {
    for (int s = steps - 1; s >= 0; --s) {
      const unsigned h16 = 16u << s;
#pragma unroll
      for (int i = 0; i < NU; ++i) {
        const float key = *reinterpret_cast<const float*>(nb + s16[i] + h16 - 16u);
        s16[i] += key < u[i] ? h16 : 0u;
      }
    }
#pragma unroll
    for (int i = 0; i < NU; ++i) off[i] = s16[i] >> 2;
  }
}

// psi_l(u), l = 0..L-1, on the segment at byte offset `off` (4 seg) of a node table.
template <typename RowT, int L, int NSEG>
__device__ __forceinline__ void pwl_eval_off(const PwlLdsN<RowT, L, NSEG>& t, unsigned off, float floor, float u,
                                             float (&y)[L]) {
  constexpr unsigned kRow = sizeof(t.seg[0]);
  const char* row = reinterpret_cast<const char*>(&t.seg[0][0]) + __umul24(off, kRow / 4);
  if constexpr (PwlLdsN<RowT, L, NSEG>::kHalf) {
    static_assert(kRow % 16 == 0 && L % 4 == 0, "rows of whole 16-byte channel quads");
    typedef __attribute__((ext_vector_type(8))) _Float16 half8_t;
    const float x = u - *reinterpret_cast<const float*>(row + 4 * L);  // the segment's anchor
#pragma unroll
    for (int q = 0; q < L / 4; ++q) {
      const half8_t v = reinterpret_cast<const half8_t*>(row)[q];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        y[4 * q + i] = relu_floor(__builtin_fmaf((float)v[2 * i], x, (float)v[2 * i + 1]), floor);
    }
  } else {
    static_assert(kRow % 16 == 0 && L % 2 == 0, "rows of whole float4 pairs");
#pragma unroll
    for (int q = 0; q < L / 2; ++q) {
      const float4 v = reinterpret_cast<const float4*>(row)[q];
      y[2 * q] = relu_floor(fmaf(v.x, u, v.y), floor);
      y[2 * q + 1] = relu_floor(fmaf(v.z, u, v.w), floor);
    }
  }
}

// Search on either table form: the node table uses its key groups when it has them.
template <int NU, int L, int NSEG>
__device__ __forceinline__ void pwl_search_any(const PwlLds<L, NSEG>& t, int steps, int, const float (&u)[NU],
                                               unsigned (&off)[NU]) {
  pwl_search_off(t, steps, u, off);
}
template <int NU, typename RowT, int L, int NSEG>
__device__ __forceinline__ void pwl_search_any(const PwlLdsN<RowT, L, NSEG>& t, int steps, int nodes,
                                               const float (&u)[NU], unsigned (&off)[NU]) {
  pwl_search_n(t, steps, nodes, u, off);
}
template <int L, int NSEG>
__device__ __forceinline__ int pwl_nodes(const PwlLds<L, NSEG>&) { return 0; }
template <typename RowT, int L, int NSEG>
__device__ __forceinline__ int pwl_nodes(const PwlLdsN<RowT, L, NSEG>& t) { return t.nodes_per_u; }

// Table type of an attention kernel: fp16 coefficients for bf16 data, fp32 otherwise.
template <typename T, int L, int NSEG>
struct PwlTab {
  using type = PwlLds<L, NSEG>;
};
template <int L, int NSEG>
struct PwlTab<__bf16, L, NSEG> {
  using type = PwlLds16<L, NSEG>;
};

// ---------------------------------------------------------------------------
// element types and fragments
// ---------------------------------------------------------------------------
template <typename T>
struct Frag;

template <>
struct Frag<__bf16> {
  bf16x8 v;
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)0.0f;
  }
  __device__ __forceinline__ void fill(float x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)x;
  }
  __device__ __forceinline__ void set(int e, float x) { v[e] = (__bf16)x; }
  // slots e and e+1 (e even) from two fp32 values: one v_cvt_pk_bf16_f32
  __device__ __forceinline__ void set2(int e, float x0, float x1) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
    const bf16x2 p = {(__bf16)x0, (__bf16)x1};
    v[e] = p[0];
    v[e + 1] = p[1];
  }
  __device__ __forceinline__ float get(int e) const { return (float)v[e]; }
};

template <>
struct Frag<float> {
  float v[8];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = 0.0f;
  }
  __device__ __forceinline__ void fill(float x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = x;
  }
  __device__ __forceinline__ void set(int e, float x) { v[e] = x; }
  __device__ __forceinline__ void set2(int e, float x0, float x1) {
    v[e] = x0;
    v[e + 1] = x1;
  }
  __device__ __forceinline__ float get(int e) const { return v[e]; }
};

__device__ __forceinline__ void mma(f32x4& c, const Frag<__bf16>& a, const Frag<__bf16>& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}

__device__ __forceinline__ void mma(f32x4& c, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
  for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[e], b.v[e], c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.0f, 0.0f, 0.0f, 0.0f}; }

// Range-checked buffers: loads past num_records bytes return 0, stores there are
// dropped, with no per-lane tests; accesses are always issued, so the waits for them
// count the same loads on every path.
constexpr int kBufferFlags = 0x00020000;  // raw 32-bit buffer, range-checked
// s_waitcnt immediate: vector memory counter 0, the others left at their maximum
constexpr int kWaitVmcnt0 = 0x0F70;

// 8 consecutive elements at byte offset `off` of a buffer
__device__ __forceinline__ void buf_load8(Frag<__bf16>& f, __amdgpu_buffer_rsrc_t rs, int off) {
  f.v = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}
__device__ __forceinline__ void buf_load8(Frag<float>& f, __amdgpu_buffer_rsrc_t rs, int off) {
  const float4 lo = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
  const float4 hi = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16, 0, 0));
  f.v[0] = lo.x; f.v[1] = lo.y; f.v[2] = lo.z; f.v[3] = lo.w;
  f.v[4] = hi.x; f.v[5] = hi.y; f.v[6] = hi.z; f.v[7] = hi.w;
}

// four consecutive elements to byte offset `off` of a buffer
template <typename T>
__device__ __forceinline__ void buf_store4(__amdgpu_buffer_rsrc_t rs, int off, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void buf_store4<__bf16>(__amdgpu_buffer_rsrc_t rs, int off, float a, float b, float c,
                                                   float d) {
  typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
  const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), rs, off, 0, 0);
}
template <>
__device__ __forceinline__ void buf_store4<float>(__amdgpu_buffer_rsrc_t rs, int off, float a, float b, float c,
                                                  float d) {
  typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, float4{a, b, c, d}), rs, off, 0, 0);
}

// Rows t0 .. t0 + nrows - 1 of a row-major [n][d] array of ESZ-byte elements as a
// range-checked buffer: rows at or past n read as 0 and are not written.  The row
// count is uniform and kept in a scalar register (a vector-held count would make
// every access a readfirstlane loop).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, int t0, int nrows, int n, int d,
                                                           int esz) {
  const char* p = reinterpret_cast<const char*>(base) + (size_t)t0 * d * esz;
  const int rows = __builtin_amdgcn_readfirstlane(max(0, min(nrows, n - t0)));
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(p), (short)0, rows * d * esz, kBufferFlags);
}

// 8 consecutive elements from memory (16 B for bf16, 32 B for fp32).
__device__ __forceinline__ void load8(Frag<__bf16>& f, const __bf16* p) {
  f.v = *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ void load8(Frag<float>& f, const float* p) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}
__device__ __forceinline__ void store8(__bf16* p, const Frag<__bf16>& f) {
  *reinterpret_cast<bf16x8*>(p) = f.v;
}
__device__ __forceinline__ void store8(float* p, const Frag<float>& f) {
  reinterpret_cast<float4*>(p)[0] = float4{f.v[0], f.v[1], f.v[2], f.v[3]};
  reinterpret_cast<float4*>(p)[1] = float4{f.v[4], f.v[5], f.v[6], f.v[7]};
}

// 4 consecutive elements from fp32 values.
__device__ __forceinline__ void store4(__bf16* p, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
  *reinterpret_cast<bf16x4*>(p) = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = float4{a, b, c, d};
}

// Load 4 consecutive elements into slots e0..e0+3 of a fragment.
__device__ __forceinline__ void load4(Frag<__bf16>& f, int e0, const __bf16* p) {
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  f.v[e0 + 0] = v[0]; f.v[e0 + 1] = v[1]; f.v[e0 + 2] = v[2]; f.v[e0 + 3] = v[3];
}
__device__ __forceinline__ void load4(Frag<float>& f, int e0, const float* p) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  f.v[e0 + 0] = v.x; f.v[e0 + 1] = v.y; f.v[e0 + 2] = v.z; f.v[e0 + 3] = v.w;
}

// Transposed operand loads.  `at(kk, col)` returns the LDS address of element
// (row k0 + kk, column c0 + col) of a logical tile in which four consecutive columns
// starting at a multiple of 4 are contiguous.  Lane (g, i) receives rows kk = 0..3
// of column i in slots e0..e0+3 (k0, c0 and the tile chosen by the caller, per lane
// group).  bf16 uses the gfx950 transpose read: within each 16-lane group, source
// lane s = 4*kk + q supplies the address of columns 4q..4q+3 of row kk and lane i
// receives column i of the four rows.  fp32 reads its four elements directly.
template <typename F>
__device__ __forceinline__ void load_tr4_at(Frag<__bf16>& f, int e0, int lane, F at) {
  const int i = lane % 16;
  typedef __attribute__((ext_vector_type(4))) short i16x4;
  const __bf16* src = at(i / 4, 4 * (i % 4));
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(__attribute__((address_space(3))) void*)(src));
  const bf16x4 b = __builtin_bit_cast(bf16x4, v);
  f.v[e0 + 0] = b[0]; f.v[e0 + 1] = b[1]; f.v[e0 + 2] = b[2]; f.v[e0 + 3] = b[3];
}
template <typename F>
__device__ __forceinline__ void load_tr4_at(Frag<float>& f, int e0, int lane, F at) {
  const int i = lane % 16;
#pragma unroll
  for (int e = 0; e < 4; ++e) f.v[e0 + e] = *at(e, i);
}

// Row-major tile X with row stride ld: rows k0..k0+3, column c0 + (lane % 16).
template <typename T>
__device__ __forceinline__ void load_tr4(Frag<T>& f, int e0, const T* X, int ld, int k0, int c0, int lane) {
  load_tr4_at(f, e0, lane, [&](int kk, int col) { return X + (size_t)(k0 + kk) * ld + c0 + col; });
}

template <typename T>
__device__ __forceinline__ T to_t(float x) { return (T)x; }

// Elements of one 16-byte vector load.
template <typename T>
struct Vec16 {
  static constexpr int N = 16 / (int)sizeof(T);
};

}  // namespace luna
