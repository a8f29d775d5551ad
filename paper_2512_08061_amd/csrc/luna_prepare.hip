// luna_prepare.hip -- exact piecewise-linear tables of the channel MLPs.
//
// The listing's channel function is psi_l(u) = relu(g_l + sum_k f_lk relu(a_lk u + c_lk))
// (outer relu when nonneg).  Every hidden unit with a_k != 0 switches state at
// beta_k = -c_k / a_k; between two consecutive breakpoints each unit is either on
// (contributes f a u + f c) or off, so the pre-activation output is s u + t there.
// Segment j is the interval (sorted[j-1], sorted[j]]; the search in the attention
// kernels returns j = number of breakpoints strictly below u.
//
// One workgroup per parameter set:
//   1. breakpoints beta_k (fp64 quotient rounded to fp32); units with a_k = 0 or a
//      non-finite quotient are constant (on iff c_k > 0) and get no breakpoint;
//   2. bitonic sort of (beta, unit) in LDS, ties broken by unit index;
//   3. the sorted breakpoints as search keys, and for every bucket of u (an
//      order-preserving partition of the reals by float bits) the start of a
//      window of 2^steps - 1 keys that holds every breakpoint a u of the bucket can
//      be compared against, steps chosen for the fullest bucket;
//   4. per channel l: segment 0 holds the units that are on below every breakpoint
//      (a < 0, or a = 0 with c > 0); crossing the breakpoint of unit k switches it on
//      (a > 0) or off (a < 0), changing (s, t) by +-(f a, f c).  The segment values
//      are these changes prefix-summed in fp64 (32 blocks per channel, block sums
//      scanned with lane shuffles), scaled by 1/sqrt(M) and rounded to fp32.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {
constexpr int kSortCap = kMaxUnits + 1;  // 1024

__device__ __forceinline__ bool key_greater(float k1, int i1, float k2, int i2) {
  return k1 > k2 || (k1 == k2 && i1 > i2);
}
}  // namespace

__global__ __launch_bounds__(256) void pwl_prepare_kernel(PrepareArgs a) {
  __shared__ float key[kSortCap];
  __shared__ int kidx[kSortCap];
  __shared__ float a_s[kSortCap], c_s[kSortCap], f_s[kSortCap];
  __shared__ int has_bp[kSortCap];
  __shared__ float g_s[16];
  __shared__ int hist[kNumBuckets];
  __shared__ float2 segv[kSegCap];  // segment values before they are written out
  __shared__ int s_vmax;            // bits of the largest |value| (non-negative float)
  __shared__ int wave_tot[4];
  __shared__ int s_nbp, s_most;

  const int set = blockIdx.x;
  const int tid = threadIdx.x;
  const int units = a.C1 * a.hidden;
  const float* A = a.fc1_w + (size_t)set * units;
  const float* Cc = a.fc1_b + (size_t)set * units;
  const float* F = a.fc2_w + (size_t)set * a.L * a.hidden;
  const float* G = a.fc2_b + (size_t)set * a.L;
  uint8_t* tab = a.tables + (size_t)set * kTableBytes;

  if (set == 0 && a.zero_ptr != nullptr)
    for (int i = tid; i < a.zero_count; i += blockDim.x) a.zero_ptr[i] = 0;
  if (tid == 0) {
    s_nbp = 0;
    s_most = 0;
    s_vmax = 0;
  }
  int N = 2;
  while (N < units) N *= 2;
  __syncthreads();

  // 1. parameters and breakpoints
  for (int k = tid; k < a.L * a.hidden; k += blockDim.x) f_s[k] = F[k];
  for (int l = tid; l < a.L; l += blockDim.x) g_s[l] = G[l];
  for (int k = tid; k < N; k += blockDim.x) {
    float bk = __builtin_inff();
    int h = 0;
    if (k < units) {
      const float ak = A[k], ck = Cc[k];
      a_s[k] = ak;
      c_s[k] = ck;
      const float q = (float)(-(double)ck / (double)ak);
      h = (ak != 0.0f) && isfinite(q);
      if (h) bk = q;
      has_bp[k] = h;
      if (h) atomicAdd(&s_nbp, 1);
    }
    key[k] = bk;
    kidx[k] = k;
  }
  __syncthreads();
  const int nbp = s_nbp;

  // 2. bitonic sort of (key, unit), ascending
  for (int size = 2; size <= N; size <<= 1) {
    for (int stride = size / 2; stride > 0; stride >>= 1) {
      for (int i = tid; i < N / 2; i += blockDim.x) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool asc = (lo & size) == 0;
        const float k1 = key[lo], k2 = key[hi];
        const int i1 = kidx[lo], i2 = kidx[hi];
        if (key_greater(k1, i1, k2, i2) == asc) {
          key[lo] = k2; key[hi] = k1;
          kidx[lo] = i2; kidx[hi] = i1;
        }
      }
      __syncthreads();
    }
  }

  // 3. search keys and bucket windows.  The sorted keys (-0 stored as +0, so that
  // bucket order and numeric order agree at zero) fall into buckets in order, so
  // the keys below bucket b are those of the buckets before it: an exclusive
  // prefix sum of the per-bucket histogram.  A u of bucket b compares against the
  // keys of bucket b only; the window must hold the fullest bucket.
  float* keys = reinterpret_cast<float*>(tab + kTabKeys);
  uint16_t* buckets = reinterpret_cast<uint16_t*>(tab + kTabBuckets);
  for (int bb = tid; bb < kNumBuckets; bb += blockDim.x) hist[bb] = 0;
  __syncthreads();
  for (int i = tid; i < nbp; i += blockDim.x) {
    const float k = key[i] == 0.0f ? 0.0f : key[i];
    key[i] = k;
    atomicAdd(&hist[bucket_of_bits(__float_as_uint(k))], 1);
  }
  __syncthreads();
  constexpr int kPer = (kNumBuckets + 255) / 256;  // buckets per thread in the scan
  int local = 0, most_local = 0;
  for (int j = 0; j < kPer; ++j) {
    const int bb = tid * kPer + j;
    if (bb < kNumBuckets) {
      local += hist[bb];
      most_local = max(most_local, hist[bb]);
    }
  }
  atomicMax(&s_most, most_local);
  // exclusive scan of the 256 per-thread totals: within 64-lane waves, then across waves
  int incl = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if ((tid & 63) >= o) incl += v;
  }
  if ((tid & 63) == 63) wave_tot[tid / 64] = incl;
  __syncthreads();
  int before = incl - local;
  for (int w = 0; w < tid / 64; ++w) before += wave_tot[w];
  const int most = s_most;
  int steps = 0;
  while ((1 << steps) - 1 < most) ++steps;
  const int window = (1 << steps) - 1;
  // +inf padding of a whole window past the last breakpoint, so that no window needs
  // shifting; only when that exceeds the capacity are late windows moved down (their
  // extra keys lie below the bucket and compare true, so counts stay exact)
  const int nkeys = nbp + window < kKeyCap ? nbp + window : kKeyCap;
  for (int j = 0; j < kPer; ++j) {
    const int bb = tid * kPer + j;
    if (bb < kNumBuckets) {
      const int start = before < nkeys - window ? before : nkeys - window;
      buckets[bb] = (uint16_t)(4 * start);
      before += hist[bb];
    }
  }
  for (int i = tid; i < nkeys; i += blockDim.x) keys[i] = i < nbp ? key[i] : __builtin_inff();

  // 4. segment values by prefix sums over the sorted breakpoints
  const double inv = 1.0 / sqrt((double)a.M);
  const int shared = (a.C1 == 1);
  const int nseg = nbp + 1;
  float vmax = 0.0f;
  const int per = (nseg + 31) / 32;  // segments per block
  const int b = tid % 32;            // block within the channel
  for (int l0 = 0; l0 < a.L; l0 += 8) {
    const int l = l0 + tid / 32;     // 32 consecutive lanes share one channel
    const bool lok = l < a.L;
    const int k0 = shared ? 0 : l * a.hidden;
    // change of (s, t) when crossing the breakpoint of rank r
    auto delta = [&](int r, double& ds, double& dt) {
      ds = 0.0;
      dt = 0.0;
      if (r >= nbp) return;
      const int k = kidx[r];
      if (k < k0 || k >= k0 + a.hidden) return;
      const double f = (double)f_s[l * a.hidden + (k - k0)];
      const double sg = a_s[k] > 0.0f ? 1.0 : -1.0;
      ds = sg * f * (double)a_s[k];
      dt = sg * f * (double)c_s[k];
    };
    // units on below every breakpoint, two per lane, reduced over the 32 lanes
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
    const int j0 = b * per, j1 = min(nseg, j0 + per);
    double ts = 0.0, tt = 0.0;
    if (lok)
      for (int r = j0; r < j1; ++r) {
        double ds, dt;
        delta(r, ds, dt);
        ts += ds;
        tt += dt;
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
      for (int j = j0; j < j1; ++j) {
        const float2 v = make_float2((float)(s * inv), (float)(t * inv));
        segv[j * a.L + l] = v;
        vmax = fmaxf(vmax, fmaxf(fabsf(v.x), fabsf(v.y)));
        double ds, dt;
        delta(j, ds, dt);
        s += ds;
        t += dt;
      }
    }
  }
  // 5. fp32 segments, and fp16 ones scaled by 2^e so that the largest magnitude
  // lands in [2^13, 2^14) (e clamped to [-20, 20])
  atomicMax(&s_vmax, __float_as_int(vmax));
  __syncthreads();
  const float vm = __int_as_float(s_vmax);
  int e = 0;
  if (vm > 0.0f && isfinite(vm)) {
    int ex;
    frexpf(vm, &ex);  // vm = m 2^ex, m in [0.5, 1)
    e = min(20, max(-20, 14 - ex));
  }
  float2* seg = reinterpret_cast<float2*>(tab + kTabSeg);
  half2_t* seg16 = reinterpret_cast<half2_t*>(tab + kTabSeg16);
  for (int i = tid; i < nseg * a.L; i += blockDim.x) {
    const float2 v = segv[i];
    seg[i] = v;
    seg16[i] = half2_t{(_Float16)ldexpf(v.x, e), (_Float16)ldexpf(v.y, e)};
  }
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
  hipLaunchKernelGGL(pwl_prepare_kernel, dim3(a.P), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace luna
