// luna_variants.hip -- feature-map variants: the template of eq. (11) of Section 3.2
// with other channel functions psi and envelopes h, as in the random-feature maps of
// Section 3.1 and the kernel ablation of Section 5.4 (Table 5).
//
//   RFF cos       sqrt(2) cos(u)                         one feature per projection
//   RFF sin/cos   (sin u, cos u)                         two
//   Performer     exp(u - |x|^2 / (2 sqrt(d)))           one (psi = exp, h = exp(-|x|^2/(2 sqrt d)))
//   MLP           Listing 1's channel MLPs with the hidden activation relu, gelu (erf
//                 form), silu or tanh, evaluated directly (a smooth activation has no
//                 piecewise-linear form), optionally gated by a tokenwise envelope
//                 sigmoid(G x + c) in [0, 1]^L (channel l of every projection), scaled
//                 per channel by Listing 1's channel RMS normalisation, and summed over
//                 the channels with global coefficients (Bank+Coef: one feature per
//                 projection)
// with u = w_i . x + b_i and every feature scaled by 1/sqrt(M).  The order is psi,
// envelope, channel RMS, bank sum, scale.
//
// One wave maps 16 rows, one workgroup 64 (the tiles of every head, a grid-stride
// loop): the projection on the matrix cores as u^T = W X^T (each lane holds four
// projections of one row), the row quantities |x|^2 and G x from the lane's slices of
// the row added across its four lane groups, then psi in fp32 registers from
// parameters in LDS.  Channel RMS needs the sums of y^2 over the whole call: a first
// pass of the same kernel accumulates them (per-workgroup fp64 partials, summed in a
// fixed order by variant_rms_kernel), the second maps with the resulting scales.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

constexpr int kVarMaxL = kVariantMaxL;
constexpr int kVarMaxHidden = 64;

__device__ __forceinline__ float var_act(int act, float z) {
  switch (act) {
    case 1: return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));  // gelu, erf form
    case 2: return z / (1.0f + expf(-z));                                 // silu
    case 3: return tanhf(z);
    default: return __builtin_elementwise_maximum(z, 0.0f);              // relu
  }
}

template <typename Tin, typename Tout, int DH>
__global__ __launch_bounds__(256) void variant_map_kernel(VariantArgs a) {
  constexpr int KS = DH / 32;
  __shared__ float s_a[kVarMaxL * kVarMaxHidden], s_c[kVarMaxL * kVarMaxHidden];
  __shared__ float s_f[kVarMaxL * kVarMaxHidden], s_g[kVarMaxL];
  __shared__ float s_env[kVarMaxL * DH], s_envb[kVarMaxL], s_bank[kVarMaxL];
  __shared__ float s_scale[kVarMaxL];
  __shared__ double s_sum[4][kVarMaxL];  // channel RMS: per-wave sums of y^2

  const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
  const int g = lane / 16, r = lane % 16;
  const int M = a.M, L = a.L, hidden = a.hidden, C1 = a.C1;
  const bool mlp = a.kind == kVarMlp;
  const int lout = mlp ? (a.bank ? 1 : L) : (a.kind == kVarSinCos ? 2 : 1);  // features per projection
  const int D = M * lout;
  const int MB = (M + 15) / 16;
  const float inv_sqrt_m = 1.0f / sqrtf((float)M);
  const float inv_2sqrt_d = 0.5f / sqrtf((float)DH);
  const int64_t n = a.rows_per_head;
  const int tiles_per_head = (int)((n + 63) / 64);
  const int64_t items = a.heads * tiles_per_head;
  float sq_acc[kVarMaxL];  // channel RMS: this thread's sums of y^2
#pragma unroll
  for (int l = 0; l < kVarMaxL; ++l) sq_acc[l] = 0.0f;

  int loaded = -1;
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t head = item / tiles_per_head;
    const int tile = (int)(item - head * tiles_per_head);
    const int hset = a.per_head ? (int)(head % a.H) : 0;
    if (hset != loaded) {  // (uniform) parameters of the set into LDS
      __syncthreads();
      if (mlp) {
        for (int i = tid; i < C1 * hidden; i += blockDim.x) {
          s_a[i] = a.fc1_w[(size_t)hset * C1 * hidden + i];
          s_c[i] = a.fc1_b[(size_t)hset * C1 * hidden + i];
        }
        for (int i = tid; i < L * hidden; i += blockDim.x) s_f[i] = a.fc2_w[(size_t)hset * L * hidden + i];
        if (tid < L) {
          s_g[tid] = a.fc2_b[(size_t)hset * L + tid];
          s_envb[tid] = a.env_b ? a.env_b[(size_t)hset * L + tid] : 0.0f;
          s_bank[tid] = a.bank ? a.bank[(size_t)hset * L + tid] : 0.0f;
          s_scale[tid] = a.rms_scale ? a.rms_scale[tid] : 1.0f;
        }
        if (a.env_w)
          for (int i = tid; i < L * DH; i += blockDim.x) s_env[i] = a.env_w[(size_t)hset * L * DH + i];
      }
      __syncthreads();
      loaded = hset;
    }
    const int64_t t = (int64_t)tile * 64 + wave * 16 + r;  // this lane's row
    const bool row_ok = t < n;
    const Tin* X = reinterpret_cast<const Tin*>(a.X) + (head * n + (row_ok ? t : 0)) * DH;
    const Tin* W = reinterpret_cast<const Tin*>(a.W) + (size_t)hset * M * DH;
    const float* bias = a.b + (size_t)hset * M;
    Tout* out = reinterpret_cast<Tout*>(a.out) + (head * n + (row_ok ? t : 0)) * (int64_t)D;
    Frag<Tin> xf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (row_ok) load8(xf[ks], X + 32 * ks + 8 * g);
      else xf[ks].zero();
    }
    // row quantities from the lane's 8 KS elements (columns 32 ks + 8 g + e), summed
    // over the row's four lane groups
    float sq = 0.0f;
    float env[kVarMaxL];
#pragma unroll
    for (int l = 0; l < kVarMaxL; ++l) env[l] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = (float)xf[ks].v[e];
        sq = fmaf(x, x, sq);
        if (mlp && a.env_w) {
          const int col = 32 * ks + 8 * g + e;
#pragma unroll
          for (int l = 0; l < kVarMaxL; ++l)
            if (l < L) env[l] = fmaf(s_env[l * DH + col], x, env[l]);
        }
      }
    sq += __shfl_xor(sq, 16, kWave);
    sq += __shfl_xor(sq, 32, kWave);
    if (mlp && a.env_w) {
#pragma unroll
      for (int l = 0; l < kVarMaxL; ++l) {
        float v = env[l];
        v += __shfl_xor(v, 16, kWave);
        v += __shfl_xor(v, 32, kWave);
        if (l < L) env[l] = 1.0f / (1.0f + expf(-(v + s_envb[l])));
      }
    }
    for (int mb = 0; mb < MB; ++mb) {
      const int prow = 16 * mb + r;  // the W row this lane feeds to the A operand
      Frag<Tin> wf[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (prow < M) load8(wf[ks], W + (size_t)prow * DH + 32 * ks + 8 * g);
        else wf[ks].zero();
      }
      f32x4 acc = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) mma(acc, wf[ks], xf[ks]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 16 * mb + 4 * g + j;  // projection of acc[j]
        if (i >= M || !row_ok) continue;
        const float u = acc[j] + bias[i];
        Tout* o = out + (int64_t)i * lout;
        if (a.kind == kVarCos) {
          o[0] = (Tout)(1.41421356237309505f * cosf(u) * inv_sqrt_m);
        } else if (a.kind == kVarSinCos) {
          o[0] = (Tout)(sinf(u) * inv_sqrt_m);
          o[1] = (Tout)(cosf(u) * inv_sqrt_m);
        } else if (a.kind == kVarPerformer) {
          o[0] = (Tout)(expf(u - sq * inv_2sqrt_d) * inv_sqrt_m);
        } else {
          float y[kVarMaxL];
#pragma unroll
          for (int l = 0; l < kVarMaxL; ++l) y[l] = 0.0f;
          if (C1 == 1) {  // one first layer: each hidden unit once, into every channel
            for (int k = 0; k < hidden; ++k) {
              const float h = var_act(a.act, fmaf(s_a[k], u, s_c[k]));
#pragma unroll
              for (int l = 0; l < kVarMaxL; ++l)
                if (l < L) y[l] = fmaf(s_f[l * hidden + k], h, y[l]);
            }
          } else {
            for (int l = 0; l < L; ++l) {  // (y[l] in registers: the channel loop is unrolled below)
              float acc_l = 0.0f;
              for (int k = 0; k < hidden; ++k)
                acc_l = fmaf(s_f[l * hidden + k], var_act(a.act, fmaf(s_a[l * hidden + k], u, s_c[l * hidden + k])),
                             acc_l);
#pragma unroll
              for (int q = 0; q < kVarMaxL; ++q)
                if (q == l) y[q] = acc_l;
            }
          }
          float sum = 0.0f;
#pragma unroll
          for (int l = 0; l < kVarMaxL; ++l) {
            if (l < L) {
              float v = y[l] + s_g[l];
              if (a.nonneg) v = __builtin_elementwise_maximum(v, 0.0f);
              if (a.env_w) v *= env[l];
              if (a.rms_pass == 1) {  // first pass of the channel RMS: sums of squares only
                sq_acc[l] = fmaf(v, v, sq_acc[l]);
              } else {
                v *= s_scale[l];
                if (a.bank) sum = fmaf(s_bank[l], v, sum);
                else o[l] = (Tout)(v * inv_sqrt_m);
              }
            }
          }
          if (a.bank && a.rms_pass != 1) o[0] = (Tout)(sum * inv_sqrt_m);
        }
      }
    }
  }
  if (a.rms_pass == 1) {  // per-workgroup sums of y^2 per channel, fp64, in a fixed order
#pragma unroll
    for (int l = 0; l < kVarMaxL; ++l) {
      double v = (double)sq_acc[l];
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
      if (lane == 0) s_sum[wave][l] = v;
    }
    __syncthreads();
    if (tid < L)
      a.rms_partial[(size_t)blockIdx.x * kVarMaxL + tid] = ((s_sum[0][tid] + s_sum[1][tid]) + s_sum[2][tid]) + s_sum[3][tid];
  }
}

// Channel RMS scales from the partials (summed in workgroup order): per channel,
// rms = sqrt(sum / count + 1e-6), scale = min(target / (rms + 1e-6), 1).
__global__ __launch_bounds__(64) void variant_rms_kernel(const double* __restrict__ partial, int groups, int L,
                                                         double count, float target, float* __restrict__ scale) {
  const int l = threadIdx.x;
  if (l >= L) return;
  double s = 0.0;
  for (int gi = 0; gi < groups; ++gi) s += partial[(size_t)gi * kVarMaxL + l];
  const double rms = sqrt(s / count + 1e-6);
  scale[l] = (float)fmin((double)target / (rms + 1e-6), 1.0);
}

template <typename Tin, typename Tout, int DH>
hipError_t variant_launch(const VariantArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((variant_map_kernel<Tin, Tout, DH>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename Tin, typename Tout>
hipError_t variant_dispatch_d(int d, const VariantArgs& a, int grid, hipStream_t s) {
  switch (d) {
    case 32: return variant_launch<Tin, Tout, 32>(a, grid, s);
    case 64: return variant_launch<Tin, Tout, 64>(a, grid, s);
    case 128: return variant_launch<Tin, Tout, 128>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void widen_kernel(const T* __restrict__ src, float* __restrict__ dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = (float)src[i];
}

}  // namespace

int variant_grid(int64_t heads, int64_t rows_per_head) {
  const int64_t items = heads * ((rows_per_head + 63) / 64);
  return (int)(items < kVariantMaxGrid ? items : kVariantMaxGrid);
}

hipError_t launch_variant_map(Dt in_dt, Dt out_dt, int d, const VariantArgs& a, hipStream_t s) {
  if (a.L > kVarMaxL || a.hidden > kVarMaxHidden) return hipErrorInvalidValue;
  const int grid = variant_grid(a.heads, a.rows_per_head);
  if (in_dt == Dt::BF16)
    return out_dt == Dt::BF16 ? variant_dispatch_d<__bf16, __bf16>(d, a, grid, s)
                              : variant_dispatch_d<__bf16, float>(d, a, grid, s);
  return out_dt == Dt::BF16 ? variant_dispatch_d<float, __bf16>(d, a, grid, s)
                            : variant_dispatch_d<float, float>(d, a, grid, s);
}

hipError_t launch_variant_rms(const double* partial, int groups, int L, double count, float target, float* scale,
                              hipStream_t s) {
  hipLaunchKernelGGL(variant_rms_kernel, dim3(1), dim3(64), 0, s, partial, groups, L, count, target, scale);
  return hipGetLastError();
}

hipError_t launch_widen(Dt dt, const void* src, float* dst, int64_t n, hipStream_t s) {
  const dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 65536)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(widen_kernel<__bf16>, grid, block, 0, s, (const __bf16*)src, dst, n);
  else hipLaunchKernelGGL(widen_kernel<float>, grid, block, 0, s, (const float*)src, dst, n);
  return hipGetLastError();
}

}  // namespace luna
