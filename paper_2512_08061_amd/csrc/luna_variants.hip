// luna_variants.hip -- launchers of the feature-map variants (kernels in
// luna_variants.hpp; those of fp32 inputs are compiled here, those of bf16 inputs in
// luna_variants_bf16.hip), the channel RMS scales and the fp32 widening of features.
#include "luna_variants.hpp"

namespace luna {

namespace {

// Channel RMS scales from the partials: per channel, rms = sqrt(sum / count + 1e-6),
// scale = min(target / (rms + 1e-6), 1).  Thread (p, l) adds the partials of groups
// p, p + 16, ... of channel l, then thread l adds the 16 sums in order: the result is
// the same on every call.
__global__ __launch_bounds__(256) void variant_rms_kernel(const double* __restrict__ partial, int groups, int L,
                                                          double count, float target, float* __restrict__ scale) {
  __shared__ double part[16][kVariantMaxL];
  const int l = threadIdx.x % kVariantMaxL, p = threadIdx.x / kVariantMaxL;
  double acc = 0.0;
  for (int gi = p; gi < groups; gi += 16) acc += partial[(size_t)gi * kVariantMaxL + l];
  part[p][l] = acc;
  __syncthreads();
  if (threadIdx.x < L) {
    double sum = 0.0;
    for (int q = 0; q < 16; ++q) sum += part[q][threadIdx.x];
    const double rms = sqrt(sum / count + 1e-6);
    scale[threadIdx.x] = (float)fmin((double)target / (rms + 1e-6), 1.0);
  }
}

// phi from the first pass's y [row][projection][channel]: y_l scale_l / sqrt(M) per
// feature, or with a bank sum_l w_l y_l scale_l / sqrt(M) per projection (the bank of
// the row's head set).  Grid-stride over the outputs, consecutive threads on
// consecutive outputs.
template <typename Tout>
__global__ __launch_bounds__(256) void variant_finish_kernel(VariantArgs a, const float* __restrict__ scale) {
  const int M = a.M, L = a.L;
  const float inv_sqrt_m = 1.0f / sqrtf((float)M);
  const int64_t rows = a.heads * a.rows_per_head;
  Tout* out = reinterpret_cast<Tout*>(a.out);
  const float* y = a.rms_y;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (a.bank) {
    const int64_t total = rows * M;
    for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < total; o += stride) {
      const int64_t row = o / M;
      const int hset = a.per_head ? (int)((row / a.rows_per_head) % a.H) : 0;
      const float* yo = y + o * L;
      const float* w = a.bank + (size_t)hset * L;
      float sum = 0.0f;
      for (int l = 0; l < L; ++l) sum = fmaf(w[l], yo[l] * scale[l], sum);
      out[o] = (Tout)(sum * inv_sqrt_m);
    }
  } else {
    const int64_t total = rows * M * L;
    for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < total; o += stride)
      out[o] = (Tout)(y[o] * scale[o % L] * inv_sqrt_m);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void widen_kernel(const T* __restrict__ src, float* __restrict__ dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = (float)src[i];
}

}  // namespace

hipError_t launch_variant_map(Dt in_dt, int d, const VariantArgs& a, int* grid, hipStream_t s) {
  if (a.kind == kVarMlp && (a.L < 1 || a.L > kVariantMaxL || a.hidden < 1)) return hipErrorInvalidValue;
  const int64_t items = a.heads * ((a.rows_per_head + 63) / 64);
  return in_dt == Dt::BF16 ? variant_map_bf16(d, a, items, grid, s) : variant_dispatch_d<float>(d, a, items, grid, s);
}

hipError_t launch_variant_finish(const VariantArgs& a, const float* scale, hipStream_t s) {
  const int64_t total = a.heads * a.rows_per_head * a.M * (a.bank ? 1 : a.L);
  const dim3 grid((unsigned)std::min<int64_t>((total + 255) / 256, 8192)), block(256);
  if (a.out_bf16) hipLaunchKernelGGL(variant_finish_kernel<__bf16>, grid, block, 0, s, a, scale);
  else hipLaunchKernelGGL(variant_finish_kernel<float>, grid, block, 0, s, a, scale);
  return hipGetLastError();
}

hipError_t launch_variant_rms(const double* partial, int groups, int L, double count, float target, float* scale,
                              hipStream_t s) {
  hipLaunchKernelGGL(variant_rms_kernel, dim3(1), dim3(256), 0, s, partial, groups, L, count, target, scale);
  return hipGetLastError();
}

hipError_t launch_widen(Dt dt, const void* src, float* dst, int64_t n, hipStream_t s) {
  const dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 65536)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(widen_kernel<__bf16>, grid, block, 0, s, (const __bf16*)src, dst, n);
  else hipLaunchKernelGGL(widen_kernel<float>, grid, block, 0, s, (const float*)src, dst, n);
  return hipGetLastError();
}

}  // namespace luna
