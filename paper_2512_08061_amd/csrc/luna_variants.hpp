// luna_variants.hpp -- feature-map variants: the template of eq. (11) of Section 3.2
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
// consecutive projections of one row), the row quantities |x|^2 and G x from the
// lane's slices of the row added across its four lane groups, then psi in fp32
// registers.  The channel MLPs' parameters are uniform across the wave and are read
// through the scalar cache into scalar registers (loads only), so that a hidden unit
// costs its two multiply-adds and its activation, and each parameter serves the lane's
// four projections.  Kernels are compiled per kind, per activation and per class of
// channel count (L <= 4, <= 8, <= 16), so that the channel values stay in registers;
// each lane writes its projections' features as one run (vector stores when the run
// is laid out as the registers hold it and aligned).
//
// Transcendentals run on the hardware units (v_exp_f32 = 2^x, v_rcp_f32, v_sin_f32 /
// v_cos_f32 of an angle in turns): exp(z) = 2^(z log2 e); sin and cos after Cody and
// Waite's reduction of u by 2 pi split into two floats, so that the hardware sees at
// most half a turn; erf by Abramowitz and Stegun's formula 7.1.26 (absolute error at
// most 1.5e-7).  Channel RMS needs the sums of y^2 over the whole call: a first pass
// of the same kernel stores y (after the envelope) in fp32 and per-workgroup fp64
// partial sums of y^2; variant_rms_kernel adds the partials in a fixed order into the
// channel scales, and variant_finish_kernel applies them, the bank sum and 1/sqrt(M).
//
// The one-feature kinds take two 16-projection blocks at a time so that a lane holds
// 8 consecutive projections (a 16-byte run of bf16 features), and read the next item's
// rows while mapping the current one.
#pragma once

#include <math.h>

#include <algorithm>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

constexpr float kLog2e = 1.44269504088896341f;
constexpr float kInvTwoPi = 0.159154943091895336f;
constexpr float kTwoPiHi = 6.28318548202514648f;   // 2 pi rounded to float
constexpr float kTwoPiLo = -1.74845553146951e-7f;  // 2 pi - kTwoPiHi

// A uniform parameter array read through the scalar cache: the constant address
// space, which the kernel only reads.
typedef const __attribute__((address_space(4))) float cfloat;
__device__ __forceinline__ cfloat* scalar_ptr(const float* p) { return (cfloat*)p; }

__device__ __forceinline__ float hw_exp(float z) { return __builtin_amdgcn_exp2f(z * kLog2e); }
__device__ __forceinline__ float hw_rcp(float z) { return __builtin_amdgcn_rcpf(z); }

// u as an angle in turns within [-1/2, 1/2]
__device__ __forceinline__ float to_turns(float u) {
  const float k = rintf(u * kInvTwoPi);
  float r = fmaf(-k, kTwoPiHi, u);
  r = fmaf(-k, kTwoPiLo, r);
  return r * kInvTwoPi;
}

// hidden activation of the channel MLPs
template <int ACT>
__device__ __forceinline__ float act_fn(float z) {
  if constexpr (ACT == 1) {  // gelu: z Phi(z) = max(z, 0) - |z| erfc(|z| / sqrt 2) / 2
    const float az = fabsf(z), x = az * 0.70710678118654752f;
    const float t = hw_rcp(fmaf(0.3275911f, x, 1.0f));
    float p = fmaf(1.061405429f, t, -1.453152027f);
    p = fmaf(p, t, 1.421413741f);
    p = fmaf(p, t, -0.284496736f);
    p = fmaf(p, t, 0.254829592f);
    const float erfc = p * t * __builtin_amdgcn_exp2f(-(x * x) * kLog2e);
    return fmaf(-0.5f * az, erfc, __builtin_elementwise_maximum(z, 0.0f));
  } else if constexpr (ACT == 2) {  // silu: z sigmoid(z)
    return z * hw_rcp(1.0f + hw_exp(-z));
  } else if constexpr (ACT == 3) {  // tanh: 1 - 2 / (e^(2z) + 1)
    return fmaf(-2.0f, hw_rcp(hw_exp(2.0f * z) + 1.0f), 1.0f);
  } else {  // relu
    return __builtin_elementwise_maximum(z, 0.0f);
  }
}

// A lane's run of RUN consecutive features (the first n valid) to out.  vec: the whole
// run with 16-byte stores (one 8-byte store for four bf16 values); the caller has
// checked the alignment.
template <int RUN>
__device__ __forceinline__ void store_run(void* out, bool obf, const float (&f)[RUN], int n, bool vec) {
  if (obf) {
    __bf16* o = reinterpret_cast<__bf16*>(out);
    if (vec && RUN == 4) {
      store4(o, f[0], f[1], f[2], f[3]);
    } else if (vec && RUN % 8 == 0) {
#pragma unroll
      for (int c = 0; c < RUN / 8; ++c) {
        bf16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (__bf16)f[8 * c + e];
        *reinterpret_cast<bf16x8*>(o + 8 * c) = v;
      }
    } else {
#pragma unroll
      for (int e = 0; e < RUN; ++e)
        if (e < n) o[e] = (__bf16)f[e];
    }
  } else {
    float* o = reinterpret_cast<float*>(out);
    if (vec && RUN % 4 == 0) {
#pragma unroll
      for (int c = 0; c < RUN / 4; ++c) store4(o + 4 * c, f[4 * c], f[4 * c + 1], f[4 * c + 2], f[4 * c + 3]);
    } else {
#pragma unroll
      for (int e = 0; e < RUN; ++e)
        if (e < n) o[e] = f[e];
    }
  }
}

// The one-feature kinds stream rows through: registers are capped so that eight waves
// per SIMD are resident (four for rows of 128 elements, which carry twice the bytes);
// the channel MLPs are bound by their arithmetic.
template <typename Tin, int DH, int KIND, int ACT, int LC, bool STAGED>
__global__ __launch_bounds__(256, KIND == kVarMlp ? 1 : (DH <= 64 ? (STAGED ? 6 : 8) : 4)) void variant_map_kernel(VariantArgs a) {
  constexpr int KS = DH / 32;
  constexpr bool MLP = KIND == kVarMlp;
  // a lane's run of features: 8 projections' (sin/cos: two each) for the one-feature
  // kinds, four projections' for the channel MLPs (with a bank; per channel otherwise)
  constexpr int RUN = MLP ? 4 : (KIND == kVarSinCos ? 16 : 8);
  __shared__ float s_bias[256];  // b of the parameter set, zero past M
  // one-feature kinds: each wave's 16 output rows (at most 256 bytes each), written back
  // as contiguous 1 KB stores
  __shared__ uint4 s_rows[STAGED ? 4 * 16 * 16 : 1];
  __shared__ float s_env[MLP ? LC * DH : 4];
  __shared__ double s_sum[4][LC];  // channel RMS: per-wave sums of y^2

  const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
  const int g = lane / 16, r = lane % 16;
  const int M = a.M, L = MLP ? a.L : 1, hidden = a.hidden;
  const bool bank = MLP && a.bank != nullptr;
  const bool env_on = MLP && a.env_w != nullptr;
  const int lout = MLP ? (bank ? 1 : L) : (KIND == kVarSinCos ? 2 : 1);  // features per projection
  const int D = M * lout;
  const int MB = (M + 15) / 16;
  const bool obf = a.out_bf16 != 0;
  const int esz = obf ? 2 : 4;
  // A run (4 lout features) goes out with vector stores when it is laid out as the
  // registers hold it (not a channel MLP with fewer channels than its class) and every
  // run start is aligned to the store width.
  const int run_bytes = (MLP ? 4 : 8) * lout * esz;
  const int chunk = min(16, run_bytes);
  const bool vec = (!MLP || bank || L == LC) && (D * esz) % chunk == 0 && run_bytes % chunk == 0 &&
                   (reinterpret_cast<uintptr_t>(a.out) & 15) == 0;
  const float inv_sqrt_m = 1.0f / sqrtf((float)M);
  const float half_inv_sqrt_d = 0.5f / sqrtf((float)DH);
  const int row_chunks = D * esz / 16;  // 16-byte pieces of an output row
  constexpr bool staged = STAGED;  // (the host checks: one-feature kind, rows of whole 16-byte pieces, <= 256 bytes)
  const int64_t n = a.rows_per_head;
  const int tiles_per_head = (int)((n + 63) / 64);
  const int64_t items = a.heads * tiles_per_head;
  float sq_acc[LC];
#pragma unroll
  for (int l = 0; l < LC; ++l) sq_acc[l] = 0.0f;

  // this lane's row of an item, as a fragment of KS 8-element slices (zeros past n)
  auto load_rows = [&](int64_t it, Frag<Tin>(&dst)[KS]) {
    const int64_t hd = it / tiles_per_head;
    const int64_t row = (it - hd * tiles_per_head) * 64 + wave * 16 + r;
    const Tin* src = reinterpret_cast<const Tin*>(a.X) + (hd * n + (row < n ? row : 0)) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (row < n) load8(dst[ks], src + 32 * ks + 8 * g);
      else dst[ks].zero();
    }
  };
  Frag<Tin> xf[KS], xnext[KS];
  if (blockIdx.x < items) load_rows(blockIdx.x, xf);

  int loaded = -1;
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t head = item / tiles_per_head;
    const int tile = (int)(item - head * tiles_per_head);
    if constexpr (!MLP) {  // the next item's rows are read while this one is mapped
      if (item + gridDim.x < items) load_rows(item + gridDim.x, xnext);
    }
    const int hset = a.per_head ? (int)(head % a.H) : 0;
    if (hset != loaded) {  // (uniform) bias and envelope weights of the set into LDS
      __syncthreads();
      s_bias[tid] = tid < M ? a.b[(size_t)hset * M + tid] : 0.0f;
      if (env_on)
        for (int i = tid; i < L * DH; i += blockDim.x) s_env[i] = a.env_w[(size_t)hset * L * DH + i];
      __syncthreads();
      loaded = hset;
    }
    const int64_t t = (int64_t)tile * 64 + wave * 16 + r;  // this lane's row
    const bool row_ok = t < n;
    const Tin* W = reinterpret_cast<const Tin*>(a.W) + (size_t)hset * M * DH;
    char* out_row = reinterpret_cast<char*>(a.out) + (head * n + (row_ok ? t : 0)) * (int64_t)D * esz;
    if constexpr (MLP) {
      if (item != blockIdx.x) load_rows(item, xf);
    }
    // row quantities from the lane's 8 KS elements (columns 32 ks + 8 g + e), summed
    // over the row's four lane groups
    float sq = 0.0f;
    if constexpr (KIND == kVarPerformer) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) sq = fmaf(xf[ks].get(e), xf[ks].get(e), sq);
      sq += __shfl_xor(sq, 16, kWave);
      sq += __shfl_xor(sq, 32, kWave);
    }
    float env[LC];
#pragma unroll
    for (int l = 0; l < LC; ++l) env[l] = 1.0f;
    if (env_on) {
#pragma unroll
      for (int l = 0; l < LC; ++l) {
        if (l < L) {
          float v = 0.0f;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const float* gw = s_env + l * DH + 32 * ks + 8 * g;
            const float4 g0 = *reinterpret_cast<const float4*>(gw);
            const float4 g1 = *reinterpret_cast<const float4*>(gw + 4);
            v = fmaf(g0.x, xf[ks].get(0), v);
            v = fmaf(g0.y, xf[ks].get(1), v);
            v = fmaf(g0.z, xf[ks].get(2), v);
            v = fmaf(g0.w, xf[ks].get(3), v);
            v = fmaf(g1.x, xf[ks].get(4), v);
            v = fmaf(g1.y, xf[ks].get(5), v);
            v = fmaf(g1.z, xf[ks].get(6), v);
            v = fmaf(g1.w, xf[ks].get(7), v);
          }
          v += __shfl_xor(v, 16, kWave);
          v += __shfl_xor(v, 32, kWave);
          env[l] = hw_rcp(1.0f + hw_exp(-(v + scalar_ptr(a.env_b)[(size_t)hset * L + l])));
        }
      }
    }
    if constexpr (!MLP) {
      // Two 16-projection blocks at a time, their W rows permuted so that lane group g
      // holds 8 consecutive projections of its row: A-operand row 4 g' + j of block bl
      // is projection 32 q + 8 g' + 4 bl + j, which the output puts in acc[bl][j] of
      // lane group g'.
      for (int q = 0; q < (M + 31) / 32; ++q) {
        const int base = 32 * q + 8 * g;  // this lane's projections base .. base + 7
        f32x4 acc[2];
#pragma unroll
        for (int bl = 0; bl < 2; ++bl) {
          const int prow = 32 * q + 8 * (r / 4) + 4 * bl + r % 4;
          Frag<Tin> wf[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            if (prow < M) load8(wf[ks], W + (size_t)prow * DH + 32 * ks + 8 * g);
            else wf[ks].zero();
          }
          acc[bl] = zero4();
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) mma(acc[bl], wf[ks], xf[ks]);
        }
        const int nv = row_ok ? max(0, min(8, M - base)) : 0;
        float f[RUN];
#pragma unroll
        for (int bl = 0; bl < 2; ++bl)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int e = 4 * bl + j;
            const float u = acc[bl][j] + s_bias[min(base + e, 255)];
            if constexpr (KIND == kVarCos) {
              f[e] = 1.41421356237309505f * inv_sqrt_m * __builtin_amdgcn_cosf(to_turns(u));
            } else if constexpr (KIND == kVarSinCos) {
              const float tu = to_turns(u);
              f[2 * e] = __builtin_amdgcn_sinf(tu) * inv_sqrt_m;
              f[2 * e + 1] = __builtin_amdgcn_cosf(tu) * inv_sqrt_m;
            } else {
              f[e] = hw_exp(u - sq * half_inv_sqrt_d) * inv_sqrt_m;
            }
          }
        if constexpr (staged) {  // the run's whole 16-byte pieces into the wave's row tile
          uint4* dst = s_rows + (wave * 16 + r) * 16 + base * lout * esz / 16;
          const int nfeat = nv * lout;
          if (obf) {
#pragma unroll
            for (int k = 0; k < RUN / 8; ++k) {
              if (8 * k < nfeat) {
                bf16x8 v;
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = (__bf16)f[8 * k + e];
                dst[k] = __builtin_bit_cast(uint4, v);
              }
            }
          } else {
#pragma unroll
            for (int k = 0; k < RUN / 4; ++k)
              if (4 * k < nfeat)
                dst[k] = make_uint4(__float_as_uint(f[4 * k]), __float_as_uint(f[4 * k + 1]),
                                    __float_as_uint(f[4 * k + 2]), __float_as_uint(f[4 * k + 3]));
          }
        } else {
          store_run<RUN>(out_row + (int64_t)base * lout * esz, obf, f, nv * lout, vec && nv == 8);
        }
      }
      if constexpr (staged) {  // the wave's 16 rows back, consecutive lanes on consecutive pieces
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        const int64_t t0 = (int64_t)tile * 64 + wave * 16;
        char* rows = reinterpret_cast<char*>(a.out) + (head * n + t0) * (int64_t)D * esz;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = lane + kWave * q;
          if (c < 16 * row_chunks) {
            const int row = c / row_chunks, col = c - row * row_chunks;
            if (t0 + row < n)
              *reinterpret_cast<uint4*>(rows + (int64_t)row * D * esz + 16 * col) = s_rows[(wave * 16 + row) * 16 + col];
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      }
    } else {
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
        const int i0 = 16 * mb + 4 * g;  // projections i0 .. i0 + 3 of row t are acc[0..3]
        const int nproj = row_ok ? max(0, min(4, M - i0)) : 0;
        float u[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) u[j] = acc[j] + s_bias[min(i0 + j, 255)];
        char* o = out_row + (int64_t)i0 * lout * esz;
        float f[RUN];
        {
          const size_t pset = (size_t)hset;
          cfloat* A = scalar_ptr(a.fc1_w + pset * a.C1 * hidden);
          cfloat* Cb = scalar_ptr(a.fc1_b + pset * a.C1 * hidden);
          cfloat* F = scalar_ptr(a.fc2_w + pset * L * hidden);
          cfloat* G = scalar_ptr(a.fc2_b + pset * L);
          float y[4][LC];
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int l = 0; l < LC; ++l) y[j][l] = 0.0f;
          if (a.C1 == 1) {  // one first layer: each hidden unit once, into every channel
#pragma unroll 4
            for (int k = 0; k < hidden; ++k) {
              const float ak = A[k], ck = Cb[k];
              float h[4];
#pragma unroll
              for (int j = 0; j < 4; ++j) h[j] = act_fn<ACT>(fmaf(ak, u[j], ck));
#pragma unroll
              for (int l = 0; l < LC; ++l) {
                if (l < L) {
                  const float fk = F[l * hidden + k];
#pragma unroll
                  for (int j = 0; j < 4; ++j) y[j][l] = fmaf(fk, h[j], y[j][l]);
                }
              }
            }
          } else {
#pragma unroll
            for (int l = 0; l < LC; ++l) {
              if (l < L) {
#pragma unroll 4
                for (int k = 0; k < hidden; ++k) {
                  const float ak = A[l * hidden + k], ck = Cb[l * hidden + k], fk = F[l * hidden + k];
#pragma unroll
                  for (int j = 0; j < 4; ++j) y[j][l] = fmaf(fk, act_fn<ACT>(fmaf(ak, u[j], ck)), y[j][l]);
                }
              }
            }
          }
          float bsum[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int l = 0; l < LC; ++l) {
            if (l < L) {
              const float gl = G[l];
              const float wl = bank ? scalar_ptr(a.bank)[pset * L + l] : 0.0f;
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                float v = y[j][l] + gl;
                if (a.nonneg) v = __builtin_elementwise_maximum(v, 0.0f);
                v *= env[l];
                if (a.rms_pass == 1) {  // sums of squares, and y kept for the second pass
                  if (j < nproj) sq_acc[l] = fmaf(v, v, sq_acc[l]);
                  y[j][l] = v;
                } else {
                    if (bank) bsum[j] = fmaf(wl, v, bsum[j]);
                  else y[j][l] = v * inv_sqrt_m;
                }
              }
            }
          }
          if (a.rms_pass == 1) {  // y in fp32, [row][projection][channel], as the second pass reads it
            char* yo = reinterpret_cast<char*>(a.rms_y) + ((head * n + (row_ok ? t : 0)) * M + i0) * (int64_t)L * 4;
            if (L == LC && nproj == 4 && (M * L) % 4 == 0) {
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                float fj[LC];
#pragma unroll
                for (int l = 0; l < LC; ++l) fj[l] = y[j][l];
                store_run<LC>(yo + (int64_t)j * LC * 4, false, fj, LC, true);
              }
            } else {
#pragma unroll
              for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int l = 0; l < LC; ++l)
                  if (j < nproj && l < L) reinterpret_cast<float*>(yo)[j * L + l] = y[j][l];
            }
          } else {
            if (bank) {
#pragma unroll
              for (int j = 0; j < 4; ++j) f[j] = bsum[j] * inv_sqrt_m;
              store_run<4>(o, obf, f, nproj, vec && nproj == 4);
            } else if (L == LC && vec && nproj == 4) {  // the run as the registers hold it: per projection
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                float fj[LC];
#pragma unroll
                for (int l = 0; l < LC; ++l) fj[l] = y[j][l];
                store_run<LC>(o + (int64_t)j * LC * esz, obf, fj, LC, true);
              }
            } else {  // element by element
#pragma unroll
              for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int l = 0; l < LC; ++l) {
                  if (j < nproj && l < L) {
                    char* p = o + (int64_t)(j * L + l) * esz;
                    if (obf) *reinterpret_cast<__bf16*>(p) = (__bf16)y[j][l];
                    else *reinterpret_cast<float*>(p) = y[j][l];
                  }
                }
            }
          }
        }
      }
    }
    if constexpr (!MLP) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) xf[ks] = xnext[ks];
    }
  }
  if constexpr (MLP) {
    if (a.rms_pass == 1) {  // per-workgroup sums of y^2 per channel, fp64, in a fixed order
#pragma unroll
      for (int l = 0; l < LC; ++l) {
        double v = (double)sq_acc[l];
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
        if (lane == 0) s_sum[wave][l] = v;
      }
      __syncthreads();
      if (tid < L)
        a.rms_partial[(size_t)blockIdx.x * kVariantMaxL + tid] =
            ((s_sum[0][tid] + s_sum[1][tid]) + s_sum[2][tid]) + s_sum[3][tid];
    }
  }
}

// As many workgroups as the device holds at once (registers and LDS permitting), at
// most kVariantMaxGrid; more items loop.  The occupancy query runs once per kernel.
template <typename Tin, int DH, int KIND, int ACT, int LC, bool STAGED = false>
hipError_t variant_launch(const VariantArgs& a, int64_t items, int* grid, hipStream_t s) {
  static const int resident = []() {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, variant_map_kernel<Tin, DH, KIND, ACT, LC, STAGED>, 256, 0) !=
            hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
    return std::min(per_cu * cus, kVariantMaxGrid);
  }();
  const int g = (int)std::min<int64_t>(items, resident);
  *grid = g;
  hipLaunchKernelGGL((variant_map_kernel<Tin, DH, KIND, ACT, LC, STAGED>), dim3(g), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename Tin, int DH>
hipError_t variant_dispatch_kind(const VariantArgs& a, int64_t items, int* grid, hipStream_t s) {
  // one-feature kinds whose output rows are whole 16-byte pieces, at most 256 bytes, at
  // an aligned address: rows staged in LDS and written back contiguously
  const int row_bytes = a.M * (a.kind == kVarSinCos ? 2 : 1) * (a.out_bf16 ? 2 : 4);
  const bool stage = row_bytes % 16 == 0 && row_bytes <= 256 && (reinterpret_cast<uintptr_t>(a.out) & 15) == 0;
  switch (a.kind) {
    case kVarCos:
      return stage ? variant_launch<Tin, DH, kVarCos, 0, 1, true>(a, items, grid, s)
                   : variant_launch<Tin, DH, kVarCos, 0, 1>(a, items, grid, s);
    case kVarSinCos:
      return stage ? variant_launch<Tin, DH, kVarSinCos, 0, 1, true>(a, items, grid, s)
                   : variant_launch<Tin, DH, kVarSinCos, 0, 1>(a, items, grid, s);
    case kVarPerformer:
      return stage ? variant_launch<Tin, DH, kVarPerformer, 0, 1, true>(a, items, grid, s)
                   : variant_launch<Tin, DH, kVarPerformer, 0, 1>(a, items, grid, s);
    case kVarMlp: break;
    default: return hipErrorInvalidValue;
  }
  const int lc = a.L <= 4 ? 0 : a.L <= 8 ? 1 : 2;
#define LUNA_VAR_MLP(ACT)                                                                  \
  case ACT:                                                                                \
    return lc == 0   ? variant_launch<Tin, DH, kVarMlp, ACT, 4>(a, items, grid, s)         \
           : lc == 1 ? variant_launch<Tin, DH, kVarMlp, ACT, 8>(a, items, grid, s)         \
                     : variant_launch<Tin, DH, kVarMlp, ACT, 16>(a, items, grid, s);
  switch (a.act) {
    LUNA_VAR_MLP(0)
    LUNA_VAR_MLP(1)
    LUNA_VAR_MLP(2)
    LUNA_VAR_MLP(3)
    default: return hipErrorInvalidValue;
  }
#undef LUNA_VAR_MLP
}

template <typename Tin>
hipError_t variant_dispatch_d(int d, const VariantArgs& a, int64_t items, int* grid, hipStream_t s) {
  switch (d) {
    case 32: return variant_dispatch_kind<Tin, 32>(a, items, grid, s);
    case 64: return variant_dispatch_kind<Tin, 64>(a, items, grid, s);
    case 128: return variant_dispatch_kind<Tin, 128>(a, items, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// the variant maps of bf16 inputs (compiled in their own translation unit)
hipError_t variant_map_bf16(int d, const VariantArgs& a, int64_t items, int* grid, hipStream_t s);

}  // namespace luna
