// luna_prepare.hip -- exact piecewise-linear tables of the channel MLPs.
//
// The listing's channel function is psi_l(u) = relu(g_l + sum_k f_lk relu(a_lk u + c_lk))
// (outer relu when nonneg).  Every hidden unit with a_k != 0 switches state at
// beta_k = -c_k / a_k; between two consecutive breakpoints each unit is either on
// (contributes f a u + f c) or off, so the pre-activation output is s u + t there.
// One workgroup per parameter set:
//   1. breakpoints beta_k (fp64 quotient rounded to fp32; units with a_k = 0 or a
//      non-finite quotient are constant: on iff c_k > 0);
//   2. stable ranks by counting (rank_k = #{beta < beta_k} + #{equal, smaller index});
//   3. heap-ordered search tree over the sorted breakpoints, padded with +inf;
//   4. per segment j and channel l: s, t summed in fp64 over the units that are on
//      inside segment j (a > 0: rank < j; a < 0: rank >= j), scaled by 1/sqrt(M),
//      rounded to fp32.
// Segment j is the interval (sorted[j-1], sorted[j]]; the search returns
// j = number of breakpoints strictly below u.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

__global__ __launch_bounds__(256) void pwl_prepare_kernel(PrepareArgs a) {
  __shared__ float beta[kMaxUnits + 1];
  __shared__ int has_bp[kMaxUnits + 1];
  __shared__ int rank[kMaxUnits + 1];
  __shared__ float sorted[kMaxUnits + 1];
  __shared__ int s_nbp;

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
  if (tid == 0) s_nbp = 0;
  __syncthreads();

  for (int k = tid; k < units; k += blockDim.x) {
    const float ak = A[k], ck = Cc[k];
    const float bk = (float)(-(double)ck / (double)ak);
    const int h = (ak != 0.0f) && isfinite(bk);
    beta[k] = bk;
    has_bp[k] = h;
    if (h) atomicAdd(&s_nbp, 1);
  }
  __syncthreads();
  const int nbp = s_nbp;

  for (int k = tid; k < units; k += blockDim.x) {
    int r = -1;
    if (has_bp[k]) {
      r = 0;
      const float bk = beta[k];
      for (int q = 0; q < units; ++q)
        r += has_bp[q] && (beta[q] < bk || (beta[q] == bk && q < k));
      sorted[r] = bk;
    }
    rank[k] = r;
  }
  __syncthreads();

  int depth = 0;
  while ((1 << depth) - 1 < nbp) ++depth;
  float* tree = reinterpret_cast<float*>(tab + kTabTree);
  for (int i = tid; i < (1 << depth); i += blockDim.x) {
    float v = __builtin_inff();
    if (i >= 1) {
      const int lv = 31 - __clz(i);          // level of heap node i (root = 0)
      const int ht = depth - 1 - lv;         // its height
      const int r = (i - (1 << lv)) * (1 << (ht + 1)) + (1 << ht) - 1;  // in-order rank
      if (r < nbp) v = sorted[r];
    }
    tree[i] = v;
  }

  const double inv = 1.0 / sqrt((double)a.M);
  const int shared = (a.C1 == 1);
  float2* seg = reinterpret_cast<float2*>(tab + kTabSeg);
  const int nseg = (nbp + 1) * a.L;
  for (int idx = tid; idx < nseg; idx += blockDim.x) {
    const int j = idx / a.L, l = idx - (idx / a.L) * a.L;
    const int k0 = shared ? 0 : l * a.hidden;
    double s = 0.0, t = (double)G[l];
    for (int kk = 0; kk < a.hidden; ++kk) {
      const int k = k0 + kk;
      const float ak = A[k], ck = Cc[k];
      const int on = has_bp[k] ? (ak > 0.0f ? (rank[k] < j) : (rank[k] >= j)) : (ck > 0.0f);
      if (on) {
        const double f = (double)F[l * a.hidden + kk];
        s += f * (double)ak;
        t += f * (double)ck;
      }
    }
    seg[idx] = make_float2((float)(s * inv), (float)(t * inv));
  }
  if (tid == 0) {
    PwlHeader* hd = reinterpret_cast<PwlHeader*>(tab + kTabHeader);
    hd->nbp = nbp;
    hd->depth = depth;
    hd->L = a.L;
    hd->nonneg = a.nonneg;
  }
}

hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(pwl_prepare_kernel, dim3(a.P), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace luna
