// luna_prepare.hip -- exact piecewise-linear tables of the channel MLPs.
//
// The channel function of the feature map is psi_l(u) = relu(g_l + sum_k f_lk relu(a_lk u + c_lk))
// (outer relu when nonneg).  Every hidden unit with a_k != 0 switches state at
// beta_k = -c_k / a_k; between two consecutive breakpoints each unit is either on
// (contributes f a u + f c) or off, so the pre-activation output is s u + t there.
// Segment j is the interval (sorted[j-1], sorted[j]]; the search in the attention
// kernels returns j = number of breakpoints strictly below u.
//
// One workgroup per parameter set:
//   1. breakpoints beta_k (fp64 quotient rounded to fp32); units with a_k = 0 or a
//      non-finite quotient are constant (on iff c_k > 0) and get no breakpoint;
//   2. a histogram of the breakpoints over the buckets of u (an order-preserving
//      partition of the reals by float bits) and its prefix sum: for every bucket
//      the start of a window of 2^steps - 1 keys that holds every breakpoint a u of
//      the bucket can be compared against, steps chosen for the fullest bucket;
//   3. the sort, as a counting sort by bucket and a rank within the bucket over the
//      distinct words (beta, unit), so ties go to the lower unit index; each
//      breakpoint is scattered to its rank with its change of (s, t);
//   4. per channel l: segment 0 holds the units that are on below every breakpoint
//      (a < 0, or a = 0 with c > 0); crossing the breakpoint of unit k switches it on
//      (a > 0) or off (a < 0), changing (s, t) by +-(f a, f c).  The segment values
//      are these changes prefix-summed in fp64 (32 blocks per channel, block sums
//      scanned with lane shuffles), scaled by 1/sqrt(M) and rounded to fp32;
//   5. the fp16 rows of the bf16 paths: per segment and channel the slope and the
//      value at the segment's anchor (its left breakpoint; the first segment's right
//      one), formed in fp64 before rounding, so that the fp16 value carries no
//      cancellation between slope u and a large intercept.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {
constexpr int kSortCap = kMaxUnits + 1;  // 1024
constexpr int kThreads = 256;
constexpr int kPadCap = kSortCap + 128;  // rank-indexed arrays, padded for whole scan blocks

// Unsigned word whose order is the float order of x (x not NaN; -0 is mapped to +0
// by the caller, so equal values give equal words).
__device__ __forceinline__ uint32_t ordered_bits(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b >> 31) ? ~b : (b | 0x80000000u);
}
}  // namespace

// SHARED: one first layer for all channels (C1 = 1), else one per channel (C1 = L)
template <bool SHARED>
__global__ __launch_bounds__(kThreads) void pwl_prepare_kernel(PrepareArgs a) {
  constexpr int kPer = (kNumBuckets + kThreads - 1) / kThreads;  // buckets per thread in the scan
  constexpr int kHist = kPer * kThreads;  // > kNumBuckets: whole runs per thread, zero counts past the end
  __shared__ unsigned long long bword[kSortCap];  // sort words grouped by bucket
  __shared__ float key[kSortCap];                  // sorted breakpoints
  __shared__ double2 dpay[kPadCap];                // per rank: change of (s, t) (see step 3)
  __shared__ int own[kPadCap];                     // per rank: owning channel, or unit (shared)
  __shared__ float a_s[kSortCap], c_s[kSortCap], f_s[kSortCap];
  __shared__ int has_bp[kSortCap];
  __shared__ float g_s[16];
  __shared__ int hist[kHist];                      // counts, then exclusive starts
  __shared__ __attribute__((aligned(16))) uint16_t bstart[(kNumBuckets + 7) / 8 * 8];
  __shared__ float2 segv[kSegCap];  // segment (slope, intercept) before they are written out
  __shared__ float segy[kSegCap];   // value at the segment's anchor
  __shared__ int s_vmax;            // bits of the largest fp16-row magnitude (non-negative float)
  __shared__ int wave_tot[kThreads / 64];
  __shared__ int s_nbp, s_most;

  const int set = blockIdx.x;
  const int tid = threadIdx.x, lane = tid % 64;
  const int units = a.C1 * a.hidden;
  const float* A = a.fc1_w + (size_t)set * units;
  const float* Cc = a.fc1_b + (size_t)set * units;
  const float* F = a.fc2_w + (size_t)set * a.L * a.hidden;
  const float* G = a.fc2_b + (size_t)set * a.L;
  uint8_t* tab = a.tables + (size_t)set * kTableBytes;

  if (tid == 0) {
    s_nbp = 0;
    s_most = 0;
    s_vmax = 0;
  }
  for (int bb = tid; bb < kHist; bb += kThreads) hist[bb] = 0;
  __syncthreads();

  // 1. parameters and breakpoints; each breakpoint is counted into its bucket, and
  // its slot there (arrival order, not deterministic) is kept for the scatter
  constexpr int kMaxPer = kSortCap / kThreads;  // units per thread
  // every load issued up front (indices clamped into the arrays; clamped values unused)
  float av[kMaxPer], cv[kMaxPer], fv[kMaxPer];
  const int nf = a.L * a.hidden;  // <= kSortCap
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m) {
    const int k = tid + kThreads * m;
    av[m] = A[min(k, units - 1)];
    cv[m] = Cc[min(k, units - 1)];
    fv[m] = F[min(k, nf - 1)];
  }
  if (tid < a.L) g_s[tid] = G[tid];
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m)
    if (tid + kThreads * m < nf) f_s[tid + kThreads * m] = fv[m];
  unsigned long long word[kMaxPer];
  float bkv[kMaxPer];  // breakpoint (+0 for -0)
  int bkt[kMaxPer], slot[kMaxPer];
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m) {
    const int k = tid + kThreads * m;
    int h = 0;
    bkt[m] = -1;
    if (k < units) {
      const float ak = av[m], ck = cv[m];
      a_s[k] = ak;
      c_s[k] = ck;
      const float q = (float)(-(double)ck / (double)ak);
      h = (ak != 0.0f) && isfinite(q);
      has_bp[k] = h;
      if (h) {
        const float bk = q == 0.0f ? 0.0f : q;
        bkv[m] = bk;
        word[m] = ((unsigned long long)ordered_bits(bk) << 32) | (unsigned)k;
        bkt[m] = bucket_of_bits(__float_as_uint(bk));
        slot[m] = atomicAdd(&hist[bkt[m]], 1);
      }
    }
    const unsigned long long hb = __ballot(h);
    if (lane == 0 && hb) atomicAdd(&s_nbp, __popcll(hb));
  }
  __syncthreads();
  const int nbp = s_nbp;

  // 2. bucket starts: exclusive prefix sum of the counts (within 64-lane waves, then
  // across waves), and the fullest bucket.  Buckets partition the reals in order, so
  // the keys below bucket b are those of the buckets before it.
  int cnt[kPer];
  int local = 0, most_local = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    cnt[j] = hist[tid * kPer + j];
    local += cnt[j];
    most_local = max(most_local, cnt[j]);
  }
  int incl = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
    most_local = max(most_local, __shfl_xor(most_local, o, 64));
  }
  if (lane == 63) wave_tot[tid / 64] = incl;
  if (lane == 0) atomicMax(&s_most, most_local);
  __syncthreads();
  int before = incl - local;
  for (int w = 0; w < tid / 64; ++w) before += wave_tot[w];
  const int most = s_most;
  int steps = 0;
  while ((1 << steps) - 1 < most) ++steps;
  const int window = (1 << steps) - 1;
  // A u of bucket b compares against the keys of bucket b only: its search window of
  // 2^steps - 1 keys starts at the bucket's first key.  The keys are padded with +inf
  // a whole window past the last breakpoint, so that no window needs shifting; only
  // when that exceeds the capacity are late windows moved down (their extra keys lie
  // below the bucket and compare true, so counts stay exact).
  const int nkeys = nbp + window < kKeyCap ? nbp + window : kKeyCap;
  // counts become exclusive starts in place (each thread owns its run of buckets);
  // the entry just past the last bucket gets nbp, the end of the last bucket
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int bb = tid * kPer + j;
    hist[bb] = before;
    if (bb < kNumBuckets) bstart[bb] = (uint16_t)(4 * (before < nkeys - window ? before : nkeys - window));
    before += cnt[j];
  }
  for (int bb = kNumBuckets + tid; bb < (kNumBuckets + 7) / 8 * 8; bb += kThreads) bstart[bb] = 0;
  __syncthreads();

  // 3. sort: every breakpoint's word goes to its bucket's range, and its rank is the
  // bucket start plus the number of words of its bucket below its own.  The words
  // (ordered key, unit index) are distinct, so the ranks are a permutation, ties
  // between equal breakpoints go to the lower unit index, and the result does not
  // depend on the arrival order.  Each breakpoint is scattered to its rank with the
  // change of (s, t) that crossing it makes, so that the segment scan reads by rank
  // without dependent lookups: per-channel first layers, f (sg a, sg c) for the
  // unit's own channel (products of two floats, exact in fp64); shared first layer,
  // (sg a, sg c), scaled per channel in the scan.  sg = sign(a).
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m)
    if (bkt[m] >= 0) bword[hist[bkt[m]] + slot[m]] = word[m];
  __syncthreads();
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m) {
    if (bkt[m] < 0) continue;
    const int k = tid + kThreads * m;
    const int b0 = hist[bkt[m]], b1 = hist[bkt[m] + 1];
    int r = b0;
    for (int j = b0; j < b1; ++j) r += (int)(bword[j] < word[m]);
    const float ak = a_s[k], ck = c_s[k];
    const double sa = ak > 0.0f ? (double)ak : -(double)ak;
    const double sc = ak > 0.0f ? (double)ck : -(double)ck;
    const double f = SHARED ? 1.0 : (double)f_s[k];
    key[r] = bkv[m];
    dpay[r] = make_double2(f * sa, f * sc);
    own[r] = SHARED ? k : k / a.hidden;
  }
  const int nseg = nbp + 1;
  const int per = ((nseg + 31) / 32 + 3) / 4 * 4;  // segments per scan block, whole groups of 4
  for (int r = nbp + tid; r < 32 * per; r += kThreads) {
    dpay[r] = make_double2(0.0, 0.0);
    own[r] = -1;
  }
  __syncthreads();
  float* keys = reinterpret_cast<float*>(tab + kTabKeys);
  for (int i = tid; i < nkeys; i += kThreads) keys[i] = i < nbp ? key[i] : __builtin_inff();

  // 4. segment values by prefix sums over the sorted breakpoints.  32 consecutive
  // lanes share one channel; lane b owns segments [b per, (b + 1) per) (ranks past
  // the last breakpoint change nothing).
  const double inv = 1.0 / sqrt((double)a.M);
  float vmax = 0.0f;
  const int b = tid % 32;  // block within the channel
  for (int l0 = 0; l0 < a.L; l0 += kThreads / 32) {
    const int l = l0 + tid / 32;
    const bool lok = l < a.L;
    const int k0 = SHARED ? 0 : l * a.hidden;
    // change of (s, t) when crossing the breakpoint of rank r
    auto delta = [&](int r, double& ds, double& dt) {
      const double2 d = dpay[r];
      const int o = own[r];
      if constexpr (SHARED) {
        const double f = o >= 0 ? (double)f_s[l * a.hidden + o] : 0.0;
        ds = f * d.x;
        dt = f * d.y;
      } else {
        ds = o == l ? d.x : 0.0;
        dt = o == l ? d.y : 0.0;
      }
    };
    // units on below every breakpoint, reduced over the 32 lanes
    double bs = 0.0, bt = 0.0;
    if (lok) {
      for (int kk = b; kk < a.hidden; kk += 32) {
        const int k = k0 + kk;
        const int on = has_bp[k] ? (a_s[k] < 0.0f) : (c_s[k] > 0.0f);
        if (on) {
          const double f = (double)f_s[l * a.hidden + kk];
          bs += f * (double)a_s[k];
          bt += f * (double)c_s[k];
        }
      }
    }
    // this block's total change
    const int j0 = b * per;
    double ts = 0.0, tt = 0.0;
    for (int i = 0; i < per; i += 4) {
      double ds[4], dt[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) delta(j0 + i + u, ds[u], dt[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ts += ds[u];
        tt += dt[u];
      }
    }
    // reductions and exclusive scans across the 32 lanes of the channel
    double es = ts, et = tt;  // inclusive scan first
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
      const double us = __shfl_up(es, o, 32), ut = __shfl_up(et, o, 32);
      if (b >= o) {
        es += us;
        et += ut;
      }
    }
    es -= ts;
    et -= tt;
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) {
      bs += __shfl_xor(bs, o, 32);
      bt += __shfl_xor(bt, o, 32);
    }
    if (lok) {
      double s = bs + es, t = (double)g_s[l] + bt + et;
      const int j1 = min(nseg, j0 + per);
      for (int i = 0; i < per && j0 + i < j1; i += 4) {
        double ds[4], dt[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) delta(j0 + i + u, ds[u], dt[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = j0 + i + u;
          if (j < j1) {
            const float2 v = make_float2((float)(s * inv), (float)(t * inv));
            segv[j * a.L + l] = v;
            const double anc = j > 0 ? (double)key[j - 1] : (nbp > 0 ? (double)key[0] : 0.0);
            const float y = (float)((s * anc + t) * inv);
            segy[j * a.L + l] = y;
            vmax = fmaxf(vmax, fmaxf(fabsf(v.x), fabsf(y)));
          }
          s += ds[u];
          t += dt[u];
        }
      }
    }
  }
  // 5. fp32 segments, and the fp16 rows scaled by 2^e so that their largest magnitude
  // lands in [2^13, 2^14).  e is clamped to [-50, 20], which keeps eps 2^(2e) a
  // normal fp32 number; magnitudes beyond 2^64, where the fp16 rows would overflow,
  // overflow fp32 in the state sums of any path as well.
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, o, 64));
  if (lane == 0) atomicMax(&s_vmax, __float_as_int(vmax));
  __syncthreads();
  const float vm = __int_as_float(s_vmax);
  int e = 0;
  if (vm > 0.0f && isfinite(vm)) {
    int ex;
    frexpf(vm, &ex);  // vm = m 2^ex, m in [0.5, 1)
    e = min(20, max(-50, 14 - ex));
  }
  {
    const uint4* src = reinterpret_cast<const uint4*>(bstart);
    uint4* dst = reinterpret_cast<uint4*>(tab + kTabBuckets);
    for (int i = tid; i < (kNumBuckets + 7) / 8; i += kThreads) dst[i] = src[i];
  }
  float2* seg = reinterpret_cast<float2*>(tab + kTabSeg);
  uint8_t* seg16 = tab + kTabSeg16;
  const int r16 = seg16_row_bytes(a.L);
  for (int i = tid; i < nseg * a.L; i += kThreads) {
    const float2 v = segv[i];
    seg[i] = v;
    const int j = i / a.L, l = i - j * a.L;
    *reinterpret_cast<half2_t*>(seg16 + (size_t)j * r16 + 4 * l) =
        half2_t{(_Float16)ldexpf(v.x, e), (_Float16)ldexpf(segy[i], e)};
  }
  for (int j = tid; j < nseg; j += kThreads)
    *reinterpret_cast<float*>(seg16 + (size_t)j * r16 + 4 * a.L) = j > 0 ? key[j - 1] : (nbp > 0 ? key[0] : 0.0f);
  if (tid == 0) {
    PwlHeader* hd = reinterpret_cast<PwlHeader*>(tab + kTabHeader);
    hd->scale_exp = e;
    hd->nbp = nbp;
    hd->steps = steps;
    hd->nkeys = nkeys;
    hd->nodes = nbp + window > kKeyCap ? 0 : (most <= 4 ? 1 : (most <= 8 ? 2 : 0));
    hd->L = a.L;
    hd->nonneg = a.nonneg;
  }
}

hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s) {
  if (a.C1 == 1) hipLaunchKernelGGL(pwl_prepare_kernel<true>, dim3(a.P), dim3(kThreads), 0, s, a);
  else hipLaunchKernelGGL(pwl_prepare_kernel<false>, dim3(a.P), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace luna
