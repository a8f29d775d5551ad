// luna_stream.hip -- one streaming step of causal LUNA attention: the prefix form of
// eq. (9) of Section 3.1 continued from a given state (S, z) over m new tokens,
//
//   for t = 0 .. m - 1:  S += phi(k_t) v_t^T,  z += phi(k_t),
//                        out_t = phi(q_t)^T S / (phi(q_t)^T z + eps),
//
// the recurrent form of the runtime section (section 4).  The features of the new
// queries and keys come from the feature-map kernel (fp32); this kernel carries the
// state.
//
// One workgroup per (head, block of 32 value columns): thread (g, j) holds S[f][j] for
// the features f = g + 8 i of its group g (interleaved, so that the eight groups read
// eight consecutive LDS words of a feature row) and the same features of z, all in
// fp32 registers for the whole step.  Per token it adds the key's outer product and
// forms its partial numerator and denominator; the eight groups' partials are summed
// through LDS in group order (deterministic), one barrier per token.  The state is
// read once at the start and written once at the end, so a step of m tokens costs one
// pass over S whatever m is.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

constexpr int kStepCols = 32;                     // value columns per workgroup
constexpr int kStepGroups = 8;                    // feature groups (threads per column)
constexpr int kStepFeat = kStepMaxD / kStepGroups;  // features per thread
constexpr int kStepTokens = 16;                   // tokens staged in LDS at a time

template <typename T>
__global__ __launch_bounds__(256) void causal_step_kernel(StepArgs a) {
  __shared__ float sq[kStepTokens][kStepMaxD];
  __shared__ float sk[kStepTokens][kStepMaxD];
  __shared__ float red[2][kStepGroups][kStepCols + 1];  // partial numerators, then the denominator

  const int nblk = a.d / kStepCols;
  const int head = blockIdx.x / nblk;
  const int cblk = blockIdx.x - head * nblk;
  const int j = threadIdx.x % kStepCols;
  const int grp = threadIdx.x / kStepCols;
  const int D = a.D, d = a.d, m = a.m;
  const int col = cblk * kStepCols + j;
  float* S = a.S + (size_t)head * D * d;
  float* z = a.z + (size_t)head * D;
  const float* PQ = a.phiq + (size_t)head * m * D;
  const float* PK = a.phik + (size_t)head * m * D;
  const T* V = reinterpret_cast<const T*>(a.V) + (size_t)head * m * d;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)head * m * d;

  float s[kStepFeat], zz[kStepFeat];
#pragma unroll
  for (int i = 0; i < kStepFeat; ++i) {
    const int f = grp + kStepGroups * i;
    s[i] = f < D ? S[(size_t)f * d + col] : 0.0f;
    zz[i] = f < D ? z[f] : 0.0f;
  }

  for (int t0 = 0; t0 < m; t0 += kStepTokens) {
    const int tn = min(kStepTokens, m - t0);
    __syncthreads();  // the previous stage's features are no longer read
    for (int idx = threadIdx.x; idx < kStepTokens * kStepMaxD; idx += blockDim.x) {
      const int tt = idx / kStepMaxD, f = idx % kStepMaxD;
      const bool ok = tt < tn && f < D;
      sq[tt][f] = ok ? PQ[(size_t)(t0 + tt) * D + f] : 0.0f;
      sk[tt][f] = ok ? PK[(size_t)(t0 + tt) * D + f] : 0.0f;
    }
    float vv[kStepTokens];
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) vv[tt] = tt < tn ? (float)V[(size_t)(t0 + tt) * d + col] : 0.0f;
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      if (tt < tn) {  // (uniform)
        float num = 0.0f, den = 0.0f;
#pragma unroll
        for (int i = 0; i < kStepFeat; ++i) {
          const int f = grp + kStepGroups * i;
          const float kf = sk[tt][f], qf = sq[tt][f];
          s[i] = fmaf(kf, vv[tt], s[i]);
          zz[i] += kf;
          num = fmaf(qf, s[i], num);
          den = fmaf(qf, zz[i], den);
        }
        const int b = (t0 + tt) & 1;  // alternating buffers: one barrier per token
        red[b][grp][j] = num;
        if (j == 0) red[b][grp][kStepCols] = den;
        __syncthreads();
        if (grp == 0) {
          float nu = 0.0f, de = 0.0f;
#pragma unroll
          for (int g2 = 0; g2 < kStepGroups; ++g2) {
            nu += red[b][g2][j];
            de += red[b][g2][kStepCols];
          }
          out[(size_t)(t0 + tt) * d + col] = (T)(nu / (de + a.eps));
        }
      }
    }
  }

#pragma unroll
  for (int i = 0; i < kStepFeat; ++i) {
    const int f = grp + kStepGroups * i;
    if (f < D) {
      S[(size_t)f * d + col] = s[i];
      if (cblk == 0 && j == 0) z[f] = zz[i];  // every column block carries the same z
    }
  }
}

}  // namespace

hipError_t launch_causal_step(Dt dt, const StepArgs& a, hipStream_t s) {
  if (a.d % kStepCols != 0 || a.D > kStepMaxD) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(a.heads * (a.d / kStepCols)));
  if (dt == Dt::BF16)
    hipLaunchKernelGGL(causal_step_kernel<__bf16>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(causal_step_kernel<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace luna
