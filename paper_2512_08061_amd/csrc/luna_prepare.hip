// luna_prepare.hip -- exact piecewise-linear tables of the channel MLPs.
//
// The channel function of the feature map is psi_l(u) = relu(g_l + sum_k f_lk relu(a_lk u + c_lk))
// (outer relu when nonneg).  Every hidden unit with a_k != 0 switches state at
// beta_k = -c_k / a_k; between two consecutive breakpoints each unit is either on
// (contributes f a u + f c) or off, so the pre-activation output is s u + t there.
// Segment j is the interval (sorted[j-1], sorted[j]]; the search in the attention
// kernels returns j = number of breakpoints strictly below u.
//
// One workgroup of 1024 threads per parameter set: a thread per hidden unit, per
// rank of the sorted breakpoints and per segment.
//   1. breakpoints beta_k (fp64 quotient rounded to fp32); units with a_k = 0 or a
//      non-finite quotient are constant (on iff c_k > 0) and get no breakpoint;
//   2. a histogram of the breakpoints over the buckets of u (an order-preserving
//      partition of the reals by float bits) and its prefix sum: for every bucket
//      the start of a window of 2^steps - 1 keys that holds every breakpoint a u of
//      the bucket can be compared against, steps chosen for the fullest bucket;
//   3. the sort, as a counting sort by bucket and a rank within the bucket over the
//      distinct words (beta, unit), so ties go to the lower unit index;
//   4. per channel l, the changes of (s, t) in the order its breakpoints are
//      crossed: crossing the breakpoint of unit k switches it on (a > 0) or off
//      (a < 0), changing (s, t) by +-(f a, f c).  With per-channel first layers a
//      unit changes only its own channel, so a channel's values are base_l plus the
//      prefix sums (fp64, one wave per channel) of its own changes, and segment j
//      takes the prefix after the channel's breakpoints ranked below j, counted by
//      one exclusive scan over the ranks of packed 8-bit per-channel counts.  With a
//      shared first layer every breakpoint changes every channel; the prefix over
//      all ranks is taken directly (at most 64 breakpoints).  base_l is g_l plus the
//      units on below every breakpoint (a < 0, or a = 0 with c > 0);
//   5. per segment (one thread each): the fp32 row of (slope, intercept) scaled by
//      1/sqrt(M), and the fp16 row of the bf16 paths: per channel the slope and the
//      value at the segment's anchor, formed in fp64 before rounding, then the anchor
//      in fp32.  The anchor is the segment's left breakpoint (the first segment's
//      right one) clamped to [-64, 64]: far breakpoints would otherwise give values
//      at the anchor that set the fp16 scale far above the channel's size where u
//      actually falls.  Any anchor gives the same function exactly; the choice only
//      bounds |slope (u - anchor)| and |value| by the channel's size on the segment.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {
constexpr int kSortCap = kMaxUnits + 1;  // 1024
constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kPer = (kNumBuckets + kThreads - 1) / kThreads;  // buckets per thread in the scan
constexpr int kMaxL = 16;
constexpr int kMaxHidden = 64;
constexpr float kAnchorMax = 64.0f;
static_assert(kPer * kThreads > kNumBuckets, "an entry past the last bucket");
static_assert(kSortCap == kThreads, "one thread per unit, rank and segment");

// Unsigned word whose order is the float order of x (x not NaN; -0 is mapped to +0
// by the caller, so equal values give equal words).
__device__ __forceinline__ uint32_t ordered_bits(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b >> 31) ? ~b : (b | 0x80000000u);
}

// Wave-wide inclusive scans on data-parallel primitives (DPP): shifts by 1, 2, 4 and 8
// within each row of 16 lanes, then the last lane of row 0 added to row 1 (and of row
// 2 to row 3), then lane 31 added to rows 2 and 3.  Lanes reading from outside their
// row get 0 (bound control), which is the identity of both operations used (sums of
// any values, maxima of non-negative values).
template <int CTRL, int ROWS>
__device__ __forceinline__ unsigned dpp32(unsigned x) {
  return (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xf, true);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp64(double x) {
  const uint2 v = __builtin_bit_cast(uint2, x);
  return __builtin_bit_cast(double, make_uint2(dpp32<CTRL, ROWS>(v.x), dpp32<CTRL, ROWS>(v.y)));
}
template <int CTRL, int ROWS, typename T>
__device__ __forceinline__ T dpp_move(T x) {
  if constexpr (sizeof(T) == 8) return dpp64<CTRL, ROWS>(x);
  else return __builtin_bit_cast(T, dpp32<CTRL, ROWS>(__builtin_bit_cast(unsigned, x)));
}
template <typename T, typename OP>
__device__ __forceinline__ T wave_scan(T x, OP op) {
  x = op(x, dpp_move<0x111, 0xf>(x));  // row_shr:1
  x = op(x, dpp_move<0x112, 0xf>(x));  // row_shr:2
  x = op(x, dpp_move<0x114, 0xf>(x));  // row_shr:4
  x = op(x, dpp_move<0x118, 0xf>(x));  // row_shr:8
  x = op(x, dpp_move<0x142, 0xa>(x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_move<0x143, 0xc>(x));  // row_bcast:31 into rows 2 and 3
  return x;
}
__device__ __forceinline__ unsigned scan_add(unsigned x) {
  return wave_scan(x, [](unsigned a, unsigned b) { return a + b; });
}
__device__ __forceinline__ double scan_add(double x) {
  return wave_scan(x, [](double a, double b) { return a + b; });
}
// the value of lane 63 (the total of an inclusive scan), in every lane
__device__ __forceinline__ unsigned last_lane(unsigned x) { return (unsigned)__builtin_amdgcn_readlane((int)x, 63); }
__device__ __forceinline__ double last_lane(double x) {
  const uint2 v = __builtin_bit_cast(uint2, x);
  return __builtin_bit_cast(double, make_uint2(last_lane(v.x), last_lane(v.y)));
}
// maximum over the wave of non-negative values (int or float bits order alike)
__device__ __forceinline__ unsigned wave_max_nonneg(unsigned x) {
  return last_lane(wave_scan(x, [](unsigned a, unsigned b) { return a > b ? a : b; }));
}

// Sum of a per-wave value over the waves below wave `wave`, from lane w holding wave
// w's value (lanes at or past kWaves hold anything): one masked scan instead of a
// dependent LDS read per wave.
__device__ __forceinline__ unsigned sum_waves_below(unsigned x, int lane, int wave) {
  return (unsigned)__builtin_amdgcn_readlane((int)scan_add(lane < wave ? x : 0u), kWaves - 1);
}

__device__ __forceinline__ unsigned pack_half2(float lo, float hi) {
  return __builtin_bit_cast(unsigned, half2_t{(_Float16)lo, (_Float16)hi});
}
}  // namespace

// SHARED: one first layer for all channels (C1 = 1), else one per channel (C1 = L)
template <bool SHARED>
__global__ __launch_bounds__(kThreads) void pwl_prepare_kernel(PrepareArgs a) {
  __shared__ unsigned long long bword[kSortCap];  // sort words grouped by bucket
  __shared__ float key[kSortCap];                  // sorted breakpoints
  __shared__ short unit_of[kSortCap];              // unit of each rank
  __shared__ int rank_of[kSortCap];                // rank of each unit's breakpoint, -1: none
  __shared__ float a_s[kSortCap], c_s[kSortCap], f_s[kSortCap];
  __shared__ int hist[kPer * kThreads];            // counts, then exclusive starts
  __shared__ __attribute__((aligned(16))) uint16_t bstart[(kNumBuckets + 7) / 8 * 8];
  // per rank r: the number of breakpoints of each channel ranked below r, 8 bits per
  // channel (channels 0-7, then 8-15); a channel has at most 64
  __shared__ unsigned long long cnt[2][kSortCap];
  __shared__ double2 dsd[kMaxL][kMaxHidden];       // per channel: its changes in crossing order
  __shared__ double2 dlt[kSortCap];                // per rank: the change its crossing makes
  __shared__ double2 cs[kMaxL][kMaxHidden + 1];    // per channel: (s, t) after p crossings
  __shared__ int wave_tot[kWaves];
  __shared__ unsigned long long wave_cnt[2][kWaves];
  __shared__ float g_s[kMaxL];
  __shared__ int s_nbp, s_most, s_vmax;

  const int set = blockIdx.x;
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int L = a.L, hidden = a.hidden;
  const int units = a.C1 * hidden;
  const int nf = L * hidden;
  const float* A = a.fc1_w + (size_t)set * units;
  const float* Cc = a.fc1_b + (size_t)set * units;
  const float* F = a.fc2_w + (size_t)set * nf;
  const float* G = a.fc2_b + (size_t)set * L;
  uint8_t* tab = a.tables + (size_t)set * kTableBytes;

  // 1. parameters (every load issued up front, indices clamped into the arrays)
  const float ak = A[min(tid, units - 1)], ck = Cc[min(tid, units - 1)];
  const float fk = F[min(tid, nf - 1)], gk = G[min(tid, L - 1)];
  if (tid == 0) {
    s_nbp = 0;
    s_most = 0;
    s_vmax = 0;
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) hist[tid + i * kThreads] = 0;
  if (tid < nf) f_s[tid] = fk;
  if (tid < L) g_s[tid] = gk;
  __syncthreads();

  // breakpoints, counted into their buckets (the slot in the bucket is arrival order)
  const int k = tid;
  int bkt = -1, slot = 0;
  unsigned long long word = 0;
  float bk = 0.0f;
  if (k < units) {
    a_s[k] = ak;
    c_s[k] = ck;
    rank_of[k] = -1;
    const float q = (float)(-(double)ck / (double)ak);
    if (ak != 0.0f && isfinite(q)) {
      bk = q == 0.0f ? 0.0f : q;
      word = ((unsigned long long)ordered_bits(bk) << 32) | (unsigned)k;
      bkt = bucket_of_bits(__float_as_uint(bk));
      slot = atomicAdd(&hist[bkt], 1);
    }
  }
  const unsigned long long hb = __ballot(bkt >= 0);
  if (lane == 0 && hb) atomicAdd(&s_nbp, __popcll(hb));
  __syncthreads();
  const int nbp = s_nbp;

  // 2. bucket starts: exclusive prefix sum of the counts (each thread a run of kPer
  // buckets, then waves, then across waves), and the fullest bucket
  int cb[kPer];
  int local = 0, most_local = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    cb[j] = hist[tid * kPer + j];
    local += cb[j];
    most_local = max(most_local, cb[j]);
  }
  const int incl = (int)scan_add((unsigned)local);
  most_local = (int)wave_max_nonneg((unsigned)most_local);
  if (lane == kWave - 1) wave_tot[wave] = incl;
  if (lane == 0) atomicMax(&s_most, most_local);
  __syncthreads();
  int before = incl - local + (int)sum_waves_below((unsigned)wave_tot[lane % kWaves], lane, wave);
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
  // counts become exclusive starts in place; the entry just past the last bucket
  // gets nbp, the end of the last bucket
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int bb = tid * kPer + j;
    hist[bb] = before;
    if (bb < kNumBuckets) bstart[bb] = (uint16_t)(4 * (before < nkeys - window ? before : nkeys - window));
    before += cb[j];
  }
  if (tid < (kNumBuckets + 7) / 8 * 8 - kNumBuckets) bstart[kNumBuckets + tid] = 0;
  __syncthreads();

  // 3. sort: every breakpoint's word goes to its bucket's range, and its rank is the
  // bucket start plus the number of words of its bucket below its own.  The words
  // (ordered key, unit index) are distinct, so the ranks are a permutation, ties
  // between equal breakpoints go to the lower unit index, and the result does not
  // depend on the arrival order.
  if (bkt >= 0) bword[hist[bkt] + slot] = word;
  __syncthreads();
  if (bkt >= 0) {
    const int b0 = hist[bkt], b1 = hist[bkt + 1];
    int r = b0;
    for (int j = b0; j < b1; ++j) r += (int)(bword[j] < word);
    key[r] = bk;
    unit_of[r] = (short)k;
    rank_of[k] = r;
    if constexpr (!SHARED) {  // per-channel first layers: f is this unit's own (fk)
      const double f = (double)fk;
      dlt[r] = make_double2(f * (ak > 0.0f ? (double)ak : -(double)ak), f * (ak > 0.0f ? (double)ck : -(double)ck));
    }
  }
  __syncthreads();

  // 4. per-channel prefix sums of the changes of (s, t)
  if constexpr (!SHARED) {
    // exclusive scan over the ranks of one-hot 8-bit channel counts
    // (8-bit fields never carry: a channel has at most 64 breakpoints, so the four
    // 32-bit words of the two counts scan independently)
    const int r = tid;
    int ch = 0;
    unsigned one[4] = {0u, 0u, 0u, 0u};
    if (r < nbp) {
      ch = unit_of[r] / hidden;
      one[ch >> 2] = 1u << (8 * (ch & 3));
    }
    unsigned ex[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const unsigned inc = scan_add(one[q]);
      ex[q] = inc - one[q];
      if (lane == kWave - 1) reinterpret_cast<unsigned*>(&wave_cnt[q >> 1][wave])[q & 1] = inc;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q)
      ex[q] += sum_waves_below(reinterpret_cast<const unsigned*>(&wave_cnt[q >> 1][lane % kWaves])[q & 1], lane, wave);
    cnt[0][r] = ((unsigned long long)ex[1] << 32) | ex[0];
    cnt[1][r] = ((unsigned long long)ex[3] << 32) | ex[2];
    // the change of each breakpoint, at its place in its channel's order
    if (r < nbp) {
      const int p = (int)((ex[ch >> 2] >> (8 * (ch & 3))) & 0xff);
      dsd[ch][p] = dlt[r];
    }
    __syncthreads();
    if (wave < L) {
      const int l = wave;
      const unsigned long long tot = cnt[l >> 3][nbp];  // every rank is below nbp
      const int nbl = (int)((tot >> (8 * (l & 7))) & 0xff);
      double bs = 0.0, bt = 0.0;
      if (lane < hidden) {
        const int u = l * hidden + lane;
        const int on = rank_of[u] >= 0 ? (a_s[u] < 0.0f) : (c_s[u] > 0.0f);
        if (on) {
          const double f = (double)f_s[u];
          bs = f * (double)a_s[u];
          bt = f * (double)c_s[u];
        }
      }
      bs = last_lane(scan_add(bs));
      bt = last_lane(scan_add(bt));
      bt += (double)g_s[l];
      const double2 dv = lane < nbl ? dsd[l][lane] : make_double2(0.0, 0.0);
      const double is = scan_add(dv.x), it = scan_add(dv.y);
      cs[l][lane + 1] = make_double2(bs + is, bt + it);
      if (lane == 0) cs[l][0] = make_double2(bs, bt);
    }
  } else {
    // one first layer: at most 64 breakpoints, each changing every channel
    if (wave < L) {
      const int l = wave;
      double bs = 0.0, bt = 0.0;
      if (lane < hidden) {
        const int on = rank_of[lane] >= 0 ? (a_s[lane] < 0.0f) : (c_s[lane] > 0.0f);
        if (on) {
          const double f = (double)f_s[l * hidden + lane];
          bs = f * (double)a_s[lane];
          bt = f * (double)c_s[lane];
        }
      }
      bs = last_lane(scan_add(bs));
      bt = last_lane(scan_add(bt));
      bt += (double)g_s[l];
      double ds = 0.0, dt = 0.0;
      if (lane < nbp) {
        const int u = unit_of[lane];
        const float au = a_s[u], cu = c_s[u];
        const double f = (double)f_s[l * hidden + u];
        ds = f * (au > 0.0f ? (double)au : -(double)au);
        dt = f * (au > 0.0f ? (double)cu : -(double)cu);
      }
      const double is = scan_add(ds), it = scan_add(dt);
      cs[l][lane + 1] = make_double2(bs + is, bt + it);
      if (lane == 0) cs[l][0] = make_double2(bs, bt);
    }
  }
  __syncthreads();

  // 5. rows, one thread per segment j: the fp32 row now, the fp16 row once the scale
  // (from the largest fp16-row magnitude) is known; both from the channel prefixes
  const int nseg = nbp + 1;
  const int j = tid;
  const double inv = 1.0 / sqrt((double)a.M);
  float anc = 0.0f, vmax = 0.0f;
  unsigned long long c0 = 0, c1 = 0;
  if (j < nseg) {
    anc = j > 0 ? key[j - 1] : (nbp > 0 ? key[0] : 0.0f);
    anc = fminf(fmaxf(anc, -kAnchorMax), kAnchorMax);
    if constexpr (!SHARED) {
      c0 = cnt[0][j];
      c1 = cnt[1][j];
    }
  }
  // (s, t) of channel l on segment j, in fp64, before the 1/sqrt(M) scale
  auto seg_st = [&](int l) {
    const int c = SHARED ? j : (int)(((l < 8 ? c0 : c1) >> (8 * (l & 7))) & 0xff);
    return cs[l][c];
  };
  if (j < nseg) {
    float2* row = reinterpret_cast<float2*>(tab + kTabSeg) + (size_t)j * L;
    for (int l = 0; l < L; l += 2) {
      const double2 v0 = seg_st(l);
      const float s0 = (float)(v0.x * inv), t0 = (float)(v0.y * inv);
      const float y0 = (float)((v0.x * (double)anc + v0.y) * inv);
      vmax = fmaxf(vmax, fmaxf(fabsf(s0), fabsf(y0)));
      if (l + 1 < L) {
        const double2 v1 = seg_st(l + 1);
        const float s1 = (float)(v1.x * inv), t1 = (float)(v1.y * inv);
        const float y1 = (float)((v1.x * (double)anc + v1.y) * inv);
        vmax = fmaxf(vmax, fmaxf(fabsf(s1), fabsf(y1)));
        if (L % 2 == 0) {  // rows of whole 16-byte pieces
          *reinterpret_cast<float4*>(row + l) = make_float4(s0, t0, s1, t1);
        } else {
          row[l] = make_float2(s0, t0);
          row[l + 1] = make_float2(s1, t1);
        }
      } else {
        row[l] = make_float2(s0, t0);
      }
    }
  }
  vmax = __uint_as_float(wave_max_nonneg(__float_as_uint(vmax)));
  if (lane == 0) atomicMax(&s_vmax, __float_as_int(vmax));
  // keys, bucket windows and header meanwhile
  {
    float* keys = reinterpret_cast<float*>(tab + kTabKeys);
    if (tid < nkeys) keys[tid] = tid < nbp ? key[tid] : __builtin_inff();
    const uint4* src = reinterpret_cast<const uint4*>(bstart);
    uint4* dst = reinterpret_cast<uint4*>(tab + kTabBuckets);
    if (tid < (kNumBuckets + 7) / 8) dst[tid] = src[tid];
    // every bucket's first comparison key (keys past the breakpoints are +inf)
    float* first = reinterpret_cast<float*>(tab + kTabFirst);
    for (int b = tid; b < kNumBuckets; b += kThreads) {
      float fk = 0.0f;
      if (steps > 0) {
        const int i = bstart[b] / 4 + (1 << (steps - 1)) - 1;
        fk = i < nbp ? key[i] : __builtin_inff();
      }
      first[b] = fk;
    }
  }
  __syncthreads();
  // The fp16 rows are scaled by 2^e so that their largest magnitude lands in
  // [2^13, 2^14).  e is clamped to [-50, 20], which keeps eps 2^(2e) a normal fp32
  // number; magnitudes beyond 2^64, where the rows would overflow, overflow fp32 in
  // the state sums of any path as well.
  const float vm = __int_as_float(s_vmax);
  int e = 0;
  if (vm > 0.0f && isfinite(vm)) {
    int ex;
    frexpf(vm, &ex);  // vm = m 2^ex, m in [0.5, 1)
    e = min(20, max(-50, 14 - ex));
  }
  if (j < nseg) {
    // words of the row: L (slope, value) half2 pairs, the anchor, zero padding; in
    // 16-byte pieces of four words
    const int r16 = seg16_row_bytes(L);
    uint4* row = reinterpret_cast<uint4*>(tab + kTabSeg16 + (size_t)j * r16);
    auto word = [&](int w) -> unsigned {
      if (w < L) {
        const double2 v = seg_st(w);
        return pack_half2(ldexpf((float)(v.x * inv), e), ldexpf((float)((v.x * (double)anc + v.y) * inv), e));
      }
      return w == L ? __float_as_uint(anc) : 0u;
    };
    for (int q = 0; 16 * q < r16; ++q) row[q] = make_uint4(word(4 * q), word(4 * q + 1), word(4 * q + 2), word(4 * q + 3));
  }
  if (tid == 0) {
    PwlHeader* hd = reinterpret_cast<PwlHeader*>(tab + kTabHeader);
    hd->scale_exp = e;
    hd->nbp = nbp;
    hd->steps = steps;
    hd->nkeys = nkeys;
    hd->nodes = nbp + window > kKeyCap ? 0 : (most <= 4 ? 1 : (most <= 8 ? 2 : 0));
    hd->L = L;
    hd->nonneg = a.nonneg;
  }
}

hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s) {
  if (a.L > kMaxL || a.hidden > kMaxHidden || a.C1 * a.hidden > kSortCap - 1) return hipErrorInvalidValue;
  if (a.C1 == 1) hipLaunchKernelGGL(pwl_prepare_kernel<true>, dim3(a.P), dim3(kThreads), 0, s, a);
  else hipLaunchKernelGGL(pwl_prepare_kernel<false>, dim3(a.P), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace luna
